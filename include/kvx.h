/*
 * kvx.h -- paged KV-cache gather / scatter / transfer for MI355X (gfx950).
 *
 * These calls are the data movement under Omni-Flow's Data Flow layer.
 * - Sec. 4.1.1 (Physical Paging Layer): a KV cache is addressed as the
 *   Cartesian product layer x page x slice, and the paging layer owns the
 *   cross-tier copy primitives.
 * - Sec. 4.1.2 (Multi-Tier Slot Engine): migration converts between the
 *   paged GPU layout and a flat per-request serialization.
 * - Sec. 5.2 (Holistic KV-Cache Takeover): the data plane translates slots
 *   to page ids.
 * - Sec. 4.1.4 (Copy-on-Write and Fragmented Page Handling): a partial
 *   write leaves the rest of its page as it was.
 *
 * Definition.  Take a request record r and a token offset i with
 * 0 <= i < n_tokens.  The element at (layer l, kv c, position
 * src_start + i, head h, dim d) of the source is copied to
 * (l, c, dst_start + i, h, d) of the destination.
 * - A pool side resolves position q through its page table:
 *       page = table[pt_off + q / page_tokens],  slot = q % page_tokens
 * - A buffer side holds the request's block [layer][kv][token][head][dim],
 *   which starts at element buf_off and is indexed by i.
 * - No other destination byte is written, and the source is only read.
 * - Elements are opaque words of elem_bytes bytes, copied bit for bit.
 *
 * Ownership.
 * - The caller owns every buffer, table, record array, error word and
 *   stream.
 * - The library allocates no device or host memory and keeps no state
 *   between calls other than a thread-local error message.
 * - Page tables and request records must be readable by the device: device
 *   memory, or pinned host memory mapped for the device.
 * - The error word must be device memory.  Bits are OR-ed into it with
 *   device atomics, which pinned host memory does not support on every
 *   platform; a host error word is refused with KVX_ERR_RANGE.
 * - Every pointer must lie in an allocation that holds the bytes the call
 *   may touch from it: kvx_pool_bytes(pool) for a pool, capacity_elems
 *   elements for a buffer, pt_len entries for a page table, n_reqs records,
 *   4 bytes for the error word.  Where the HIP runtime reports the
 *   allocation around a pointer (every device allocation), a shorter one
 *   is refused with KVX_ERR_RANGE before anything is enqueued.
 * - Device memory must belong to the current device (hipGetDevice); memory
 *   of another GPU is refused with KVX_ERR_RANGE.  Kernels run on the
 *   current device.
 * - Descriptors are read on the host during the call.
 *
 * Synchrony.
 * - The entry points enqueue kernels on `stream` (a hipStream_t; NULL is
 *   the default stream) and return without waiting.
 * - Destination data and *dev_err are valid once the stream has
 *   synchronised.
 *
 * Errors.
 * - A call returns KVX_OK or a negative kvx_status, with nothing enqueued.
 *   kvx_last_error() then names the failing check.
 * - Problems that only the device can see skip the affected elements and
 *   OR bits into *dev_err (when non-NULL; kvx_page_hashes requires it):
 *   - KVX_DERR_SRC_PAGE / KVX_DERR_DST_PAGE: a page id outside
 *     [0, num_pages);
 *   - KVX_DERR_PT_RANGE: a table index outside [0, pt_len);
 *   - KVX_DERR_BAD_REQ: a malformed request record.  The whole record is
 *     skipped.
 *   - KVX_DERR_BAD_PLAN (kvx_transfer_planned only): the plan disagrees
 *     with the records;
 *   - KVX_DERR_STALLED (kvx_page_hashes only): the chain of a group waited
 *     longer than its bound for a digest and gave up; outputs of that group
 *     are incomplete.  The bound is far beyond any digest time, so this
 *     indicates a defect in the library, not in the input.  A build with
 *     the macro KVX_HASH_IDLE_POLLS defined uses that many empty polls as
 *     the bound instead; the test build sets 1 to force the case.
 * - The destination side is resolved before the source side, so a
 *   position bad on both sides reports only the destination bit.
 * - Source and destination may be the same pool.  Copy-on-write of shared
 *   pages (Sec. 4.1.4) copies pages into fresh pages of the same pool.  The
 *   result is defined as long as no element the call writes is also read by
 *   it.
 * - Not detected: two records that write the same destination slot, and an
 *   element that one call both reads and writes.  Both give undefined
 *   results.
 */
#ifndef KVX_H
#define KVX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVX_ABI_VERSION 1

/* Most request records per call (each workgroup of the copy kernel reads
 * the whole record array, 256 records at a time). */
#define KVX_MAX_REQS 65536
/* Largest page (tokens) a pool may declare. */
#define KVX_MAX_PAGE_TOKENS (1 << 20)

/* Memory order of a pool.  The letters name axes outermost first:
 * L layer, P page, C kv component, T token slot, H head, D head_dim.
 * D is innermost in every layout, so a (l, p, c, t, h) "row" of
 * head_dim * elem_bytes bytes is always contiguous. */
typedef enum kvx_layout {
    KVX_LPCTHD = 0, /* [layer][page][kv][token][head][dim]: the NHD block stack */
    KVX_LPCHTD = 1, /* [layer][page][kv][head][token][dim] */
    KVX_PLCTHD = 2, /* [page][layer][kv][token][head][dim] */
    KVX_PLCHTD = 3  /* [page][layer][kv][head][token][dim] */
} kvx_layout;

typedef enum kvx_status {
    KVX_OK = 0,
    KVX_ERR_NULL = -1,      /* a required pointer is NULL */
    KVX_ERR_SHAPE = -2,     /* sides differ in layers/kv/heads/head_dim/elem_bytes,
                               or a dimension is out of range */
    KVX_ERR_ALIGN = -3,     /* a base pointer, or head_dim * elem_bytes, is not a
                               multiple of 16 bytes */
    KVX_ERR_LAYOUT = -4,    /* unknown layout, or num_kv not 1 or 2 */
    KVX_ERR_RANGE = -5,     /* n_reqs, pt_len or a size out of range */
    KVX_ERR_HIP = -6        /* the HIP runtime refused a query or a launch */
} kvx_status;

/* Device-side error bits. */
#define KVX_DERR_SRC_PAGE 1u
#define KVX_DERR_DST_PAGE 2u
#define KVX_DERR_PT_RANGE 4u
#define KVX_DERR_BAD_REQ 8u
#define KVX_DERR_STALLED 16u
#define KVX_DERR_BAD_PLAN 32u

/* A paged pool of num_pages pages; element (l, p, c, t, h, d) lives where
 * `layout` puts it.  `base` is device memory (or device-mapped pinned host
 * memory), 16-byte aligned, and must hold kvx_pool_bytes(pool) bytes (a
 * smaller allocation is refused where the runtime reports its size, see
 * Ownership above). */
typedef struct kvx_pool {
    void *base;
    int32_t num_layers;  /* L >= 1 */
    int32_t num_kv;      /* C: 2 (K and V) or 1 (one latent, as in MLA) */
    int32_t num_heads;   /* H >= 1 */
    int32_t head_dim;    /* D >= 1; D * elem_bytes a multiple of 16 */
    int32_t page_tokens; /* T, 1 .. KVX_MAX_PAGE_TOKENS */
    int32_t num_pages;   /* N >= 1 */
    int32_t elem_bytes;  /* 1, 2, 4 or 8 */
    int32_t layout;      /* a kvx_layout */
} kvx_pool;

/* A flat buffer of per-request blocks [layer][kv][token][head][dim] (the
 * flat serialization used by host tiers).  `base` is device memory or
 * device-mapped pinned host memory, 16-byte aligned, and must hold
 * capacity_elems elements (checked as for a pool).
 * With capacity_elems == 0 `base` may be NULL: only records of 0 tokens at
 * offset 0 then fit, and any other record raises KVX_DERR_BAD_REQ. */
typedef struct kvx_buf {
    void *base;
    int32_t num_layers, num_kv, num_heads, head_dim, elem_bytes;
    int32_t reserved;        /* 0 */
    int64_t capacity_elems;  /* elements addressable from base */
} kvx_buf;

/* One request record (40 bytes).  A record is malformed (KVX_DERR_BAD_REQ)
 * if n_tokens < 0, a start is negative, a start + n_tokens exceeds
 * 2^31 - 1, `reserved` is not 0, or, for a buffer side, its start is not 0
 * or its block [buf_off, buf_off + L*C*n_tokens*H*D) is not 16-byte aligned
 * or does not fit the buffer. */
typedef struct kvx_req {
    int64_t src_pt_off; /* index in src_pt of the request's logical page 0 */
    int64_t dst_pt_off; /* index in dst_pt of the request's logical page 0 */
    int64_t buf_off;    /* element offset of the request's block (buffer side) */
    int32_t src_start;  /* first position read (0 for a buffer source) */
    int32_t dst_start;  /* first position written (0 for a buffer destination) */
    int32_t n_tokens;   /* positions moved; 0 moves nothing */
    int32_t reserved;   /* must be 0 */
} kvx_req;

/* Pool -> pool, with any change of page size and layout.
 * Sec. 4.1 (role-to-role sharing through the Global Params Pool); Sec. 5.1
 * (partial-prefix reuse: src_start/dst_start select [p, len)).
 * src_pt / dst_pt: int32 page tables of src_pt_len / dst_pt_len entries.
 * reqs: n_reqs records (0 <= n_reqs <= KVX_MAX_REQS). */
int kvx_transfer(const kvx_pool *src, const kvx_pool *dst,
                 const int32_t *src_pt, int64_t src_pt_len,
                 const int32_t *dst_pt, int64_t dst_pt_len,
                 const kvx_req *reqs, int32_t n_reqs,
                 uint32_t *dev_err, void *stream);

/* A layer range, a kv range and a head range, each at its own offset on
 * either side (40 bytes).  Sec. 4.1.1: a view names a tuple of layers and a
 * tuple of slices; Sec. 4.1.3: one node may hold the K half of a page and
 * another the V half; Sec. 7: transfers between tensor-parallel layouts
 * (a head range) and pipeline stages (a layer range). */
typedef struct kvx_slice {
    int32_t src_layer0, dst_layer0, num_layers;
    int32_t src_kv0, dst_kv0, num_kv;
    int32_t src_head0, dst_head0, num_heads;
    int32_t reserved; /* must be 0 */
} kvx_slice;

/* Slice of a pool -> slice of another pool.  For every request record r,
 * 0 <= i < n_tokens, l < num_layers, c < num_kv, h < num_heads and every d:
 *   dst(dst_layer0 + l, dst_kv0 + c, dst_start + i, dst_head0 + h, d)
 *     := src(src_layer0 + l, src_kv0 + c, src_start + i, src_head0 + h, d)
 * The pools may differ in num_layers, num_kv and num_heads (and page size,
 * page count and layout); head_dim and elem_bytes must match (else
 * KVX_ERR_SHAPE).  Each range must lie inside its pool, counts must be
 * >= 0 (KVX_ERR_RANGE otherwise); a zero count enqueues nothing.  Every
 * other rule, argument and device error bit is that of kvx_transfer, which
 * is this call with all ranges full and equal shapes. */
int kvx_transfer_slice(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                       const int32_t *src_pt, int64_t src_pt_len,
                       const int32_t *dst_pt, int64_t dst_pt_len,
                       const kvx_req *reqs, int32_t n_reqs,
                       uint32_t *dev_err, void *stream);

/* Layer-pipelined pool -> pool transfer (Sec. 7: hierarchical transmission;
 * Sec. 5.1: pipelined prefill).  The copied layers (all of them when `slice`
 * is NULL, else the slice's layer range) are moved in consecutive groups of
 * layers_per_group layers, one launch per group, in order, on `stream`.
 * After group g the call records events[g] on `stream`.  A consumer stream
 * that waits on events[g] may use those layers of the destination while
 * later groups are still moving.
 * - events: hipEvent_t handles created by the caller (the library creates
 *   none); n_events must be >= the number of groups.
 * - Every event is recorded even when nothing is copied.  If a launch
 *   fails, the call returns KVX_ERR_HIP, and the events of that group and
 *   later groups are not recorded.
 * - The data result equals kvx_transfer_slice / kvx_transfer with the same
 *   arguments. */
int kvx_transfer_layered(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                         const int32_t *src_pt, int64_t src_pt_len,
                         const int32_t *dst_pt, int64_t dst_pt_len,
                         const kvx_req *reqs, int32_t n_reqs,
                         int32_t layers_per_group, void *const *events, int32_t n_events,
                         uint32_t *dev_err, void *stream);

/* Pool -> flat buffer: the offload (serialization) direction of Sec. 4.1.2. */
int kvx_gather(const kvx_pool *src, const kvx_buf *dst,
               const int32_t *src_pt, int64_t src_pt_len,
               const kvx_req *reqs, int32_t n_reqs,
               uint32_t *dev_err, void *stream);

/* Flat buffer -> pool: the onload direction of Sec. 4.1.2. */
int kvx_scatter(const kvx_buf *src, const kvx_pool *dst,
                const int32_t *dst_pt, int64_t dst_pt_len,
                const kvx_req *reqs, int32_t n_reqs,
                uint32_t *dev_err, void *stream);

/* Slice of a pool -> flat buffer that holds exactly the slice (Sec. 4.1.2
 * migration of a Sec. 4.1.1 view: offload only V, a layer range, or one
 * tensor-parallel head range).  For every record r, token i < n_tokens,
 * l < num_layers, c < num_kv, h < num_heads and every d:
 *   block_r(l, c, i, h, d)
 *     := src(src_layer0 + l, src_kv0 + c, src_start + i, src_head0 + h, d)
 * where block_r is the record's block [num_layers][num_kv][n_tokens]
 * [num_heads][head_dim] at buf_off.
 * - The buffer's num_layers, num_kv and num_heads must equal the slice's
 *   counts (KVX_ERR_SHAPE otherwise), its head_dim and elem_bytes the
 *   pool's; the slice's destination offsets must be 0 and its source range
 *   must lie inside the pool (KVX_ERR_RANGE otherwise).
 * - Every other rule, argument and device error bit is kvx_gather's, which
 *   is this call with the full slice. */
int kvx_gather_slice(const kvx_pool *src, const kvx_buf *dst, const kvx_slice *slice,
                     const int32_t *src_pt, int64_t src_pt_len,
                     const kvx_req *reqs, int32_t n_reqs,
                     uint32_t *dev_err, void *stream);

/* Flat buffer that holds exactly a slice -> that slice of a pool (the onload
 * of kvx_gather_slice):
 *   dst(dst_layer0 + l, dst_kv0 + c, dst_start + i, dst_head0 + h, d)
 *     := block_r(l, c, i, h, d)
 * The slice's source offsets must be 0 and its destination range must lie
 * inside the pool; otherwise as kvx_gather_slice and kvx_scatter. */
int kvx_scatter_slice(const kvx_buf *src, const kvx_pool *dst, const kvx_slice *slice,
                      const int32_t *dst_pt, int64_t dst_pt_len,
                      const kvx_req *reqs, int32_t n_reqs,
                      uint32_t *dev_err, void *stream);

/* One destination page of a planned transfer (32 bytes): where request
 * `req` writes its page jj, that is, the tokens [dst_slot, dst_slot +
 * n_tokens) of destination page dst_pt[dst_idx], read from the source page
 * src_pt[src_idx] from slot src_slot on (and on into the following source
 * pages).  Indices outside the int32 range are stored clamped to it. */
typedef struct kvx_plan_slot {
    int32_t dst_idx;    /* index in dst_pt of the page */
    int32_t src_idx;    /* index in src_pt of the page holding the first token */
    int32_t dst_slot;   /* first slot written in the page */
    int32_t n_tokens;   /* tokens written in the page, >= 1 */
    int32_t src_slot;   /* slot of the first token in its source page */
    int32_t req;        /* the record */
    int32_t reserved[2];
} kvx_plan_slot;

/* Bytes of a plan of n_reqs records and plan_pages destination pages. */
#define KVX_PLAN_BYTES(n_reqs, plan_pages) (((int64_t)(n_reqs) + 1) * 8 + (int64_t)(plan_pages) * 32)

/* kvx_transfer / kvx_transfer_slice (slice NULL: everything) with a plan,
 * for callers that build their records on the host.  The plan spells out,
 * page by page, the work the records imply, so that the kernel copying a
 * piece of a page finds it with one read instead of a search:
 * plan: device memory (or mapped pinned host memory), KVX_PLAN_BYTES bytes,
 *   8-byte aligned, written by kvx_plan_fill():
 *   - int64 prefix[n_reqs + 1]: the exclusive prefix over the records of
 *     the destination pages each touches, pages(r) = (dst_start + n_tokens
 *     - 1) / T_dst - dst_start / T_dst + 1 for a well-formed record with
 *     n_tokens > 0, else 0 (a malformed record, as in the kvx_req rules,
 *     counts 0);
 *   - kvx_plan_slot slots[plan_pages], in record order, page order within
 *     a record.
 * plan_pages: prefix[n_reqs]; plan_tokens: n_tokens summed over the
 *   well-formed records (kvx_plan_pages returns both).  Read on the host to
 *   shape the launch.
 * When the records copy at least 64 KiB per destination page and layer on
 * average and both tables hold at most INT32_MAX entries, the call can
 * sweep: one workgroup per 1 KiB piece of each destination page of each
 * layer, layer by layer and page by page, every page on one XCD, instead of
 * a persistent grid.  Started in that order by the hardware, the pieces in
 * flight stay within a small window that slides through the transfer; on
 * MI355X this holds the handoff's 256 KiB pages at 6.1-6.35 TB/s and MLA's
 * 72 KiB pages at 5.75-5.97 TB/s in every process, where the persistent grid
 * ranges from 5.1 to 6.4 TB/s with the physical placement of the pools
 * (for MLA above the sweep in most processes, 3-8% below it in others).
 * Which of the two launches such a call takes follows
 * kvx_set_launch_choice(): by default the faster one on these pools, found
 * by timing both on the first calls.
 * Otherwise the call runs as the unplanned one and the plan is not read.
 * Results, error bits and every rule are those of kvx_transfer(_slice):
 * - a plan that disagrees with the records, or with the pools' page sizes,
 *   raises KVX_DERR_BAD_PLAN, and the destination is then defined only
 *   where the plan and the records agree (every access still stays inside
 *   the pools and tables); plan_pages other than prefix[n_reqs] is such a
 *   disagreement;
 * - a wrong plan_tokens changes only the choice of launch.
 * plan_pages or plan_tokens < 0, a NULL plan with n_reqs > 0, or a plan
 * extent below KVX_PLAN_BYTES is refused on the host. */
int kvx_transfer_planned(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                         const int32_t *src_pt, int64_t src_pt_len,
                         const int32_t *dst_pt, int64_t dst_pt_len,
                         const kvx_req *reqs, int32_t n_reqs,
                         const void *plan, int64_t plan_pages, int64_t plan_tokens,
                         uint32_t *dev_err, void *stream);

/* kvx_transfer_layered with a plan: each layer group's launch is that of
 * kvx_transfer_planned over the group's layers (the plan describes pages,
 * so one plan serves every group).  Arguments, events and rules are those
 * of kvx_transfer_layered and kvx_transfer_planned; the plan is checked
 * against the records in every group's launch. */
int kvx_transfer_layered_planned(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                                 const int32_t *src_pt, int64_t src_pt_len,
                                 const int32_t *dst_pt, int64_t dst_pt_len,
                                 const kvx_req *reqs, int32_t n_reqs,
                                 int32_t layers_per_group, void *const *events, int32_t n_events,
                                 const void *plan, int64_t plan_pages, int64_t plan_tokens,
                                 uint32_t *dev_err, void *stream);

/* How a kvx_transfer_planned call that can sweep picks its launch.  Both
 * launches write the same bytes; which is faster depends on where the pools
 * sit in physical memory, and that does not change while they live.
 * - KVX_CHOOSE_MEASURED (the default): per key (device, both pool base
 *   pointers and descriptors, and the slice: the pair of pools, whatever
 *   the records of each call) the first six calls take the sweep and the
 *   persistent grid in turn,
 *   untimed (the first calls on fresh pools run slow, whichever launch they
 *   take); the next four are timed between HIP events, in the order sweep,
 *   grid, grid, sweep, so that a drift that remains weighs on both launches
 *   alike.  Once all four have completed (polled with hipEventQuery, never
 *   waited on) every later call takes the launch that moved more tokens
 *   (plan_tokens) per millisecond over its two timed calls.  Until then
 *   calls sweep.  Calls made while their
 *   stream is being captured record no events: they take the key's decided
 *   launch, else the sweep, and do not count.  Eight HIP events per key in
 *   measurement are the only resources this takes (no device memory); at
 *   most 64 keys are kept, the least recently used dropped first.  A caller
 *   that frees its pools and gets new ones at the same addresses keeps the
 *   old decision until the next kvx_set_launch_choice().
 * - KVX_CHOOSE_SWEEP: always the sweep.
 * - KVX_CHOOSE_GRID: always the persistent grid.
 * kvx_transfer_layered_planned sweeps every group whenever the sweep can
 * serve it, except under KVX_CHOOSE_GRID.  The setting is process-wide;
 * setting it (to any mode) forgets every key.  Returns KVX_OK, or
 * KVX_ERR_RANGE for another value. */
#define KVX_CHOOSE_MEASURED 0
#define KVX_CHOOSE_SWEEP 1
#define KVX_CHOOSE_GRID 2
int kvx_set_launch_choice(int mode);

/* The current KVX_CHOOSE_* mode. */
int kvx_launch_choice(void);

/* Launch kinds reported by kvx_last_launch(). */
#define KVX_LAUNCH_NONE 0   /* the call enqueued no kernel */
#define KVX_LAUNCH_GRID 1   /* the persistent grid */
#define KVX_LAUNCH_SWEEP 2  /* the sweep */

/* The kind of the last kernel the calling thread's last copy call
 * (transfer, gather or scatter, any variant) enqueued. */
int kvx_last_launch(void);

/* Sizes a plan from a host copy of the records: writes the exclusive prefix
 * of pages per record into prefix[0..n_reqs] and the tokens of the
 * well-formed records into *tokens (each if not NULL), and returns the
 * total of pages, for the side `side` (0: source positions, 1: destination
 * positions) of a pool with page_tokens tokens per page.  -1 on bad
 * arguments. */
int64_t kvx_plan_pages(const kvx_req *host_reqs, int32_t n_reqs, int32_t page_tokens, int32_t side,
                       int64_t *prefix, int64_t *tokens);

/* Writes the plan of kvx_transfer_planned for these records and page sizes
 * into host memory `plan` of KVX_PLAN_BYTES(n_reqs, plan_pages) bytes,
 * 8-byte aligned; plan_pages must be the total kvx_plan_pages returns for
 * side 1 and dst_page_tokens.  KVX_ERR_RANGE on bad arguments or a
 * plan_pages that differs from that total, KVX_ERR_NULL / KVX_ERR_ALIGN for
 * the pointers. */
int kvx_plan_fill(const kvx_req *host_reqs, int32_t n_reqs, int32_t src_page_tokens,
                  int32_t dst_page_tokens, int64_t plan_pages, void *plan);

/* One chained-hash request (32 bytes). */
typedef struct kvx_hash_req {
    int64_t payload_off;  /* first position of the request in the payload */
    int64_t out_off;      /* index in `out` of the hash of the request's page 0 */
    uint64_t seed;        /* chain state before page 0: 0 for a new chain, or the
                             hash of the last full page of the prefix it extends */
    int32_t n_positions;  /* positions of the request; 0 hashes nothing */
    int32_t reserved;     /* must be 0 */
} kvx_hash_req;

/* Chained page hashes (Sec. 5.1: each page's hash encodes its predecessor's,
 * so hashes are equal only when the whole prefix matches page by page).
 * The paper names no hash function.  The definition used, with fnv =
 * FNV-1a 64 (offset basis 0xcbf29ce484222325, prime 0x100000001b3):
 *   page j of request r = its positions [j*T, min((j+1)*T, n)) of records
 *                         of rec_bytes bytes (token ids, modality digests);
 *   c_j = fnv(bytes of page j)
 *   h_j = fnv(le64(h_{j-1}) || le64(c_j)),   h_{-1} = seed
 *   out[out_off + j] = h_j for j < ceil(n / T).
 * payload: device memory (or mapped pinned host memory), 4-byte aligned,
 * payload_positions records.  rec_bytes: a positive multiple of 4.
 * page_tokens: 1 .. KVX_MAX_PAGE_TOKENS.  out: out_len uint64 words,
 * 8-byte aligned; requests must not share output words, and out must not
 * overlap the payload.  The call enqueues one kernel, which writes the page
 * digests c_j into out and replaces each with h_j once h_{j-1} is known, so
 * out holds final values only once the stream has passed the kernel.
 * A record whose positions or outputs fall outside the arrays, with
 * n_positions < 0 or a nonzero reserved word, is skipped (its outputs are
 * not written) and raises KVX_DERR_BAD_REQ.
 * dev_err is required (KVX_ERR_NULL when NULL): KVX_DERR_STALLED is the
 * only sign that a group's outputs were left incomplete. */
int kvx_page_hashes(const void *payload, int64_t payload_positions, int32_t rec_bytes,
                    int32_t page_tokens, const kvx_hash_req *reqs, int32_t n_reqs,
                    uint64_t *out, int64_t out_len, uint32_t *dev_err, void *stream);

/* Bytes a pool described by *pool occupies (-1 if the descriptor is invalid). */
int64_t kvx_pool_bytes(const kvx_pool *pool);

/* Static text for a kvx_status value. */
const char *kvx_strerror(int status);

/* The calling thread's message for its last failed call ("" if none). */
const char *kvx_last_error(void);

/* KVX_ABI_VERSION of the loaded library. */
int kvx_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVX_H */
