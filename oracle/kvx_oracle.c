/*
 * kvx_oracle.c -- CPU oracle for the paged KV-cache gather / scatter /
 * transfer path.  TEST INFRASTRUCTURE ONLY: tests, the smoke check and the
 * benchmark's CPU-baseline leg call it; the product path never does.
 *
 * What is computed (Omni-Flow, Sec. 4.1.1 "Physical Paging Layer" and
 * Sec. 4.1.2 "Multi-Tier Slot Engine"; Sec. 4.1.4 for partial pages):
 *
 *   The KV cache of a model is a Cartesian product layer x page x slice
 *   (Sec. 4.1.1), where a page holds T consecutive token positions of one
 *   request and a slice is one (K-or-V, head) buffer whose innermost extent
 *   is head_dim.  A request's logical token position q lives in the page
 *   named by its page table at entry floor(q / T), at slot q mod T (the
 *   slot-to-page translation the data plane owns, Sec. 5.2 "Holistic
 *   KV-Cache Takeover").  Migration between tiers converts between a paged
 *   GPU layout and a flat per-request serialization (Sec. 4.1.2).
 *
 *   For every request r and every i in [0, n_r):
 *       ps = src_start_r + i   (position read)
 *       pd = dst_start_r + i   (position written)
 *   and every (layer l, kv c, head h, dim d):
 *       DST(l, c, pd, h, d) := SRC(l, c, ps, h, d)
 *   where a pool side resolves a position through its page table and a
 *   buffer side addresses the request's block [layer][kv][token][head][dim]
 *   with the buffer token index i.  Nothing else in the destination changes
 *   (a partial page keeps its other slots, Sec. 4.1.4 "Copy-on-Write and
 *   Fragmented Page Handling"), and the source is only read.
 *
 * Elements are opaque e-byte words copied byte by byte; they never pass
 * through a floating-point register.
 *
 * Defined error behaviour (the same rules the library documents): a request
 * record that is malformed is skipped and raises ORA_ERR_BAD_REQ; a position
 * whose page-table index falls outside the table raises ORA_ERR_PT_RANGE and
 * is skipped; a page id outside [0, num_pages) raises ORA_ERR_SRC_PAGE or
 * ORA_ERR_DST_PAGE and is skipped.  The destination side is resolved before
 * the source side.
 *
 * Plain C, no shared code with the GPU library.  Loop order r, i, l, c, h, d.
 */
#include <stdint.h>

enum {
    ORA_LPCTHD = 0, /* [layer][page][kv][token][head][dim] */
    ORA_LPCHTD = 1, /* [layer][page][kv][head][token][dim] */
    ORA_PLCTHD = 2, /* [page][layer][kv][token][head][dim] */
    ORA_PLCHTD = 3  /* [page][layer][kv][head][token][dim] */
};

enum {
    ORA_ERR_SRC_PAGE = 1,
    ORA_ERR_DST_PAGE = 2,
    ORA_ERR_PT_RANGE = 4,
    ORA_ERR_BAD_REQ = 8
};

/* Shape of a paged pool: layers, kv components, heads, head_dim, tokens per
 * page, pages, bytes per element, layout code. */
typedef struct {
    int64_t L, C, H, D, T, N, e, layout;
} ora_pool;

/* Shape of a flat buffer holding per-request blocks
 * [layer][kv][token][head][dim]; cap = elements addressable. */
typedef struct {
    int64_t L, C, H, D, e, cap;
} ora_buf;

/* Element index of (layer l, kv c, page p, slot s, head h, dim d). */
static int64_t pool_index(const ora_pool *P, int64_t l, int64_t c, int64_t p,
                          int64_t s, int64_t h, int64_t d)
{
    switch (P->layout) {
    case ORA_LPCTHD:
        return ((((l * P->N + p) * P->C + c) * P->T + s) * P->H + h) * P->D + d;
    case ORA_LPCHTD:
        return ((((l * P->N + p) * P->C + c) * P->H + h) * P->T + s) * P->D + d;
    case ORA_PLCTHD:
        return ((((p * P->L + l) * P->C + c) * P->T + s) * P->H + h) * P->D + d;
    case ORA_PLCHTD:
        return ((((p * P->L + l) * P->C + c) * P->H + h) * P->T + s) * P->D + d;
    }
    return -1;
}

/* Element index of (layer l, kv c, token i, head h, dim d) in the block of a
 * request holding n tokens that starts at element off. */
static int64_t buf_index(const ora_buf *B, int64_t off, int64_t n, int64_t l,
                         int64_t c, int64_t i, int64_t h, int64_t d)
{
    return off + (((l * B->C + c) * n + i) * B->H + h) * B->D + d;
}

static void copy_elem(uint8_t *dst, const uint8_t *src, int64_t e)
{
    for (int64_t b = 0; b < e; ++b)
        dst[b] = src[b];
}

/* Resolve position q of a paged side to (page, slot).  Returns 0 on success,
 * else the error bit that applies. */
static int resolve(const ora_pool *P, const int32_t *pt, int64_t pt_len,
                   int64_t pt_off, int64_t q, int page_err, int64_t *page,
                   int64_t *slot)
{
    int64_t idx = pt_off + q / P->T;
    if (idx < 0 || idx >= pt_len)
        return ORA_ERR_PT_RANGE;
    int64_t id = pt[idx];
    if (id < 0 || id >= P->N)
        return page_err;
    *page = id;
    *slot = q % P->T;
    return 0;
}

/* A request's position range [start, start + n) must be non-negative and
 * representable as 32-bit positions. */
static int range_ok(int64_t start, int64_t n)
{
    return n >= 0 && start >= 0 && start + n <= INT32_MAX;
}

/* A buffer block must start 16-byte aligned and fit the buffer. */
static int block_ok(const ora_buf *B, int64_t off, int64_t n)
{
    if (off < 0 || (off * B->e) % 16 != 0)
        return 0;
    return off + B->L * B->C * n * B->H * B->D <= B->cap;
}

/* Request records are rows of six int64 values:
 *   src_pt_off, dst_pt_off, buf_off, src_start, dst_start, n_tokens. */
#define R_SRC_PT 0
#define R_DST_PT 1
#define R_BUF 2
#define R_SRC_START 3
#define R_DST_START 4
#define R_N 5

/* Pool -> pool. */
uint32_t ora_transfer(const uint8_t *src, const ora_pool *S, uint8_t *dst,
                      const ora_pool *Dp, const int32_t *src_pt,
                      int64_t src_pt_len, const int32_t *dst_pt,
                      int64_t dst_pt_len, const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_SRC_START], n) || !range_ok(q[R_DST_START], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t ps = q[R_SRC_START] + i, pd = q[R_DST_START] + i;
            int64_t sp, ss, dp, ds;
            int bad = resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT], pd,
                              ORA_ERR_DST_PAGE, &dp, &ds);
            if (!bad)
                bad = resolve(S, src_pt, src_pt_len, q[R_SRC_PT], ps,
                              ORA_ERR_SRC_PAGE, &sp, &ss);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < S->L; ++l)
                for (int64_t c = 0; c < S->C; ++c)
                    for (int64_t h = 0; h < S->H; ++h)
                        for (int64_t d = 0; d < S->D; ++d)
                            copy_elem(dst + Dp->e * pool_index(Dp, l, c, dp, ds, h, d),
                                      src + S->e * pool_index(S, l, c, sp, ss, h, d),
                                      S->e);
        }
    }
    return err;
}

/* Pool -> flat buffer (offload / serialization). */
uint32_t ora_gather(const uint8_t *src, const ora_pool *S, uint8_t *dst,
                    const ora_buf *B, const int32_t *src_pt, int64_t src_pt_len,
                    const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_SRC_START], n) || q[R_DST_START] != 0 ||
            !block_ok(B, q[R_BUF], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t sp, ss;
            int bad = resolve(S, src_pt, src_pt_len, q[R_SRC_PT],
                              q[R_SRC_START] + i, ORA_ERR_SRC_PAGE, &sp, &ss);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < S->L; ++l)
                for (int64_t c = 0; c < S->C; ++c)
                    for (int64_t h = 0; h < S->H; ++h)
                        for (int64_t d = 0; d < S->D; ++d)
                            copy_elem(dst + B->e * buf_index(B, q[R_BUF], n, l, c, i, h, d),
                                      src + S->e * pool_index(S, l, c, sp, ss, h, d),
                                      S->e);
        }
    }
    return err;
}

/* Flat buffer -> pool (onload / deserialization). */
uint32_t ora_scatter(const uint8_t *src, const ora_buf *B, uint8_t *dst,
                     const ora_pool *Dp, const int32_t *dst_pt,
                     int64_t dst_pt_len, const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_DST_START], n) || q[R_SRC_START] != 0 ||
            !block_ok(B, q[R_BUF], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t dp, ds;
            int bad = resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT],
                              q[R_DST_START] + i, ORA_ERR_DST_PAGE, &dp, &ds);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < Dp->L; ++l)
                for (int64_t c = 0; c < Dp->C; ++c)
                    for (int64_t h = 0; h < Dp->H; ++h)
                        for (int64_t d = 0; d < Dp->D; ++d)
                            copy_elem(dst + Dp->e * pool_index(Dp, l, c, dp, ds, h, d),
                                      src + B->e * buf_index(B, q[R_BUF], n, l, c, i, h, d),
                                      Dp->e);
        }
    }
    return err;
}

/* Slice of a pool -> slice of another pool (Sec. 4.1.1: a view names a
 * tuple of layers and a tuple of slices; Sec. 4.1.3: one node may hold the
 * K half of a page and another the V half; Sec. 7: transfers between
 * different tensor-parallel layouts).
 *
 * sl[] = { src_layer0, dst_layer0, n_layers, src_kv0, dst_kv0, n_kv,
 *          src_head0, dst_head0, n_heads }
 * For every request r, i in [0, n_r), l < n_layers, c < n_kv, h < n_heads,
 * d < head_dim:
 *   DST(dst_layer0 + l, dst_kv0 + c, pd, dst_head0 + h, d)
 *       := SRC(src_layer0 + l, src_kv0 + c, ps, src_head0 + h, d)
 * The pools may differ in layers, kv components and heads; head_dim and
 * element size match.  Same resolution and error rules as ora_transfer. */
uint32_t ora_transfer_slice(const uint8_t *src, const ora_pool *S, uint8_t *dst,
                            const ora_pool *Dp, const int64_t *sl,
                            const int32_t *src_pt, int64_t src_pt_len,
                            const int32_t *dst_pt, int64_t dst_pt_len,
                            const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    /* A slice with no layer, kv component or head copies no element, and a
     * call that copies nothing checks nothing: no record or table is read. */
    if (sl[2] == 0 || sl[5] == 0 || sl[8] == 0)
        return 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_SRC_START], n) || !range_ok(q[R_DST_START], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t ps = q[R_SRC_START] + i, pd = q[R_DST_START] + i;
            int64_t sp, ss, dp, ds;
            int bad = resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT], pd,
                              ORA_ERR_DST_PAGE, &dp, &ds);
            if (!bad)
                bad = resolve(S, src_pt, src_pt_len, q[R_SRC_PT], ps,
                              ORA_ERR_SRC_PAGE, &sp, &ss);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < sl[2]; ++l)
                for (int64_t c = 0; c < sl[5]; ++c)
                    for (int64_t h = 0; h < sl[8]; ++h)
                        for (int64_t d = 0; d < S->D; ++d)
                            copy_elem(dst + Dp->e * pool_index(Dp, sl[1] + l, sl[4] + c, dp, ds,
                                                               sl[7] + h, d),
                                      src + S->e * pool_index(S, sl[0] + l, sl[3] + c, sp, ss,
                                                              sl[6] + h, d),
                                      S->e);
        }
    }
    return err;
}

/* Slice of a pool -> flat buffer (Sec. 4.1.2 migration restricted to a
 * view, Sec. 4.1.1: a view names a tuple of layers and a tuple of slices).
 * sl is the nine-field slice of ora_transfer_slice.  Write (L0, K0, H0)
 * for its source offsets (fields 0, 3, 6) and (nl, nk, nh) for its counts
 * (fields 2, 5, 8).  The buffer holds exactly the slice: its blocks are
 * [nl][nk][n][nh][D] (the buffer shape's L, C, H).  For every request r,
 * token i < n, layer l < nl, kv c < nk, head h < nh and every d:
 *     block_r(l, c, i, h, d) := POOL(L0 + l, K0 + c, src_start + i, H0 + h, d)
 * A slice with a zero count copies and checks nothing. */
uint32_t ora_gather_slice(const uint8_t *src, const ora_pool *S, uint8_t *dst,
                          const ora_buf *B, const int64_t *sl,
                          const int32_t *src_pt, int64_t src_pt_len,
                          const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    if (sl[2] == 0 || sl[5] == 0 || sl[8] == 0)
        return 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_SRC_START], n) || q[R_DST_START] != 0 ||
            !block_ok(B, q[R_BUF], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t sp, ss;
            int bad = resolve(S, src_pt, src_pt_len, q[R_SRC_PT],
                              q[R_SRC_START] + i, ORA_ERR_SRC_PAGE, &sp, &ss);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < sl[2]; ++l)
                for (int64_t c = 0; c < sl[5]; ++c)
                    for (int64_t h = 0; h < sl[8]; ++h)
                        for (int64_t d = 0; d < S->D; ++d)
                            copy_elem(dst + B->e * buf_index(B, q[R_BUF], n, l, c, i, h, d),
                                      src + S->e * pool_index(S, sl[0] + l, sl[3] + c,
                                                              sp, ss, sl[6] + h, d),
                                      S->e);
        }
    }
    return err;
}

/* Flat buffer -> slice of a pool: the reverse of ora_gather_slice, with
 * the pool's range starting at the slice's destination offsets (L1, K1, H1)
 * (fields 1, 4, 7):
 *     POOL(L1 + l, K1 + c, dst_start + i, H1 + h, d) := block_r(l, c, i, h, d) */
uint32_t ora_scatter_slice(const uint8_t *src, const ora_buf *B, uint8_t *dst,
                           const ora_pool *Dp, const int64_t *sl,
                           const int32_t *dst_pt, int64_t dst_pt_len,
                           const int64_t *reqs, int64_t n_reqs)
{
    uint32_t err = 0;
    if (sl[2] == 0 || sl[5] == 0 || sl[8] == 0)
        return 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 6 * r;
        int64_t n = q[R_N];
        if (!range_ok(q[R_DST_START], n) || q[R_SRC_START] != 0 ||
            !block_ok(B, q[R_BUF], n)) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t dp, ds;
            int bad = resolve(Dp, dst_pt, dst_pt_len, q[R_DST_PT],
                              q[R_DST_START] + i, ORA_ERR_DST_PAGE, &dp, &ds);
            if (bad) {
                err |= (uint32_t)bad;
                continue;
            }
            for (int64_t l = 0; l < sl[2]; ++l)
                for (int64_t c = 0; c < sl[5]; ++c)
                    for (int64_t h = 0; h < sl[8]; ++h)
                        for (int64_t d = 0; d < Dp->D; ++d)
                            copy_elem(dst + Dp->e * pool_index(Dp, sl[1] + l, sl[4] + c,
                                                               dp, ds, sl[7] + h, d),
                                      src + B->e * buf_index(B, q[R_BUF], n, l, c, i, h, d),
                                      Dp->e);
        }
    }
    return err;
}

/* ------------------------------------------------------------------------
 * Chained page hashes (Sec. 5.1 "Chained Paged Hashing": each page's hash
 * encodes the hash of its predecessor, so two hashes are equal only when the
 * whole prefix matches page by page).  The paper names no hash function;
 * the definition used here:
 *
 *   fnv(bytes, h): FNV-1a 64 (Fowler, Noll and Vo): for each byte b in
 *       order, h = (h xor b) * 0x100000001b3 mod 2^64; the empty-input state
 *       is the offset basis 0xcbf29ce484222325.
 *   Request r covers positions [off_r, off_r + n_r) of a payload of records
 *   of rec_bytes bytes (token ids, modality digests).  Page j holds its
 *   positions [j*T, min((j+1)*T, n_r)).
 *   c_j = fnv(bytes of page j, basis)                 (page digest)
 *   h_j = fnv(le64(h_{j-1}) || le64(c_j), basis)      (chain), h_{-1} = seed_r
 *   out[out_off_r + j] = h_j for j < ceil(n_r / T).
 *
 * A request continues an earlier chain by passing the hash of its last
 * full page as seed (incremental matching, Sec. 5.1).  A malformed record
 * (n < 0, positions or outputs outside the arrays) is skipped and raises
 * ORA_ERR_BAD_REQ.  Hash records are rows of four int64 values:
 *   payload_off (positions), out_off, seed (bits), n_positions.
 * ------------------------------------------------------------------------ */
#define FNV_BASIS 0xcbf29ce484222325ull
#define FNV_PRIME 0x100000001b3ull

uint64_t ora_fnv1a64(const uint8_t *p, int64_t n, uint64_t h)
{
    for (int64_t i = 0; i < n; ++i) {
        h ^= p[i];
        h *= FNV_PRIME;
    }
    return h;
}

static void le64(uint8_t *out, uint64_t v)
{
    for (int b = 0; b < 8; ++b)
        out[b] = (uint8_t)(v >> (8 * b));
}

uint32_t ora_page_hashes(const uint8_t *payload, int64_t payload_positions,
                         int64_t rec_bytes, int64_t T, const int64_t *reqs,
                         int64_t n_reqs, uint64_t *out, int64_t out_len)
{
    uint32_t err = 0;
    for (int64_t r = 0; r < n_reqs; ++r) {
        const int64_t *q = reqs + 4 * r;
        int64_t off = q[0], out_off = q[1], n = q[3];
        uint64_t h = (uint64_t)q[2];
        int64_t pages = n > 0 ? (n + T - 1) / T : 0;
        if (n < 0 || off < 0 || off + n > payload_positions || out_off < 0 ||
            out_off + pages > out_len) {
            err |= ORA_ERR_BAD_REQ;
            continue;
        }
        for (int64_t j = 0; j < pages; ++j) {
            int64_t first = j * T;
            int64_t count = (n - first < T) ? n - first : T;
            uint64_t c = ora_fnv1a64(payload + (off + first) * rec_bytes,
                                     count * rec_bytes, FNV_BASIS);
            uint8_t pair[16];
            le64(pair, h);
            le64(pair + 8, c);
            h = ora_fnv1a64(pair, 16, FNV_BASIS);
            out[out_off + j] = h;
        }
    }
    return err;
}
