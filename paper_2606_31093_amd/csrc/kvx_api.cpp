// kvx_api.cpp -- the C-ABI of libkvx (include/kvx.h): host-side validation
// of descriptors, derivation of byte strides per layout, the choice between
// the sweep and the persistent grid for planned transfers, and the launch
// of the copy kernel on the caller's stream.  No device memory is allocated
// here.

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kvx.h"
#include "kvx_hash.h"
#include "kvx_internal.h"

namespace {

thread_local std::string g_last_error;
thread_local int g_last_launch = KVX_LAUNCH_NONE;

int fail(int status, const char *fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(msg, sizeof msg, fmt, ap);
    va_end(ap);
    g_last_error = msg;
    return status;
}

// a * b for non-negative operands, or -1 if the product exceeds int64.
int64_t mul_checked(int64_t a, int64_t b) {
    if (a < 0 || b < 0) return -1;
    if (a != 0 && b > INT64_MAX / a) return -1;
    return a * b;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Element shape shared by both sides of a call.
struct Shape {
    int32_t L, C, H, D, e;
};

int check_shape(const char *name, const Shape &s) {
    if (s.L < 1 || s.H < 1 || s.D < 1)
        return fail(KVX_ERR_SHAPE, "%s: num_layers, num_heads and head_dim must be >= 1", name);
    if (s.C != 1 && s.C != 2) return fail(KVX_ERR_LAYOUT, "%s: num_kv must be 1 or 2 (got %d)", name, s.C);
    if (s.e != 1 && s.e != 2 && s.e != 4 && s.e != 8)
        return fail(KVX_ERR_SHAPE, "%s: elem_bytes must be 1, 2, 4 or 8 (got %d)", name, s.e);
    const int64_t row = (int64_t)s.D * s.e;
    if (row % 16 != 0)
        return fail(KVX_ERR_ALIGN, "%s: head_dim * elem_bytes = %lld is not a multiple of 16", name,
                    (long long)row);
    const int64_t token = mul_checked(mul_checked(mul_checked(s.L, s.C), s.H), row);
    if (token < 0 || token > (int64_t(1) << 31))
        return fail(KVX_ERR_SHAPE, "%s: one token spans more than 2 GiB across all layers", name);
    return KVX_OK;
}

int pool_shape(const kvx_pool *p, const char *name, Shape &s) {
    if (!p) return fail(KVX_ERR_NULL, "%s: pool descriptor is NULL", name);
    s = Shape{p->num_layers, p->num_kv, p->num_heads, p->head_dim, p->elem_bytes};
    int st = check_shape(name, s);
    if (st) return st;
    if (p->layout < KVX_LPCTHD || p->layout > KVX_PLCHTD)
        return fail(KVX_ERR_LAYOUT, "%s: unknown layout %d", name, p->layout);
    if (p->page_tokens < 1 || p->page_tokens > KVX_MAX_PAGE_TOKENS)
        return fail(KVX_ERR_SHAPE, "%s: page_tokens %d outside [1, %d]", name, p->page_tokens,
                    KVX_MAX_PAGE_TOKENS);
    if (p->num_pages < 1) return fail(KVX_ERR_SHAPE, "%s: num_pages must be >= 1", name);
    // A tile (one page of one layer) must stay below 2^31 16-byte vectors.
    const int64_t tile_vecs = (int64_t)s.C * p->page_tokens * s.H * (s.D * s.e / 16);
    if (tile_vecs >= (int64_t(1) << 31))
        return fail(KVX_ERR_SHAPE, "%s: one page of one layer exceeds 32 GiB", name);
    return KVX_OK;
}

int64_t pool_bytes(const kvx_pool *p) {
    int64_t b = mul_checked(mul_checked(mul_checked(p->num_layers, p->num_kv), p->num_heads),
                            (int64_t)p->head_dim * p->elem_bytes);
    b = mul_checked(mul_checked(b, p->page_tokens), p->num_pages);
    return b;
}

int same_shape(const Shape &a, const Shape &b) {
    if (a.L != b.L || a.C != b.C || a.H != b.H || a.D != b.D || a.e != b.e)
        return fail(KVX_ERR_SHAPE,
                    "source and destination differ in element shape: (L,C,H,D,e) = "
                    "(%d,%d,%d,%d,%d) vs (%d,%d,%d,%d,%d)",
                    a.L, a.C, a.H, a.D, a.e, b.L, b.C, b.H, b.D, b.e);
    return KVX_OK;
}

// The device must be able to address `ptr` (device memory or mapped pinned
// host memory), and the allocation it points into must hold the `need`
// bytes from `ptr` on that the call may touch.  On success *dev_ptr is the
// address kernels use and *is_host (if given) tells whether it is host
// memory.  With `device_only` pinned host memory is refused too.
int device_view(const void *ptr, int64_t need, const char *name, void **dev_ptr,
                bool *is_host = nullptr, bool device_only = false) {
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, ptr);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // clear the sticky error the query leaves
        return fail(KVX_ERR_RANGE, "%s (%p) is not memory the GPU can address (%s)", name, ptr,
                    hipGetErrorString(e));
    }
    const bool dev_mem = attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged ||
                         attr.type == hipMemoryTypeUnified;
    const bool host_mem = attr.type == hipMemoryTypeHost && attr.devicePointer;
    if (!dev_mem && !host_mem)
        return fail(KVX_ERR_RANGE, "%s (%p) is not device memory or mapped pinned host memory",
                    name, ptr);
    if (device_only && !dev_mem)
        return fail(KVX_ERR_RANGE, "%s (%p) must be device memory (pinned host memory is refused)",
                    name, ptr);
    if (attr.type == hipMemoryTypeDevice) {
        // Device memory of another GPU would fault the kernel unless peer
        // access happened to be enabled; this library runs on one GPU.
        int cur = 0;
        const hipError_t ge = hipGetDevice(&cur);
        if (ge != hipSuccess)
            return fail(KVX_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(ge));
        if (attr.device != cur)
            return fail(KVX_ERR_RANGE, "%s (%p) is memory of device %d, but the current device is %d",
                        name, ptr, attr.device, cur);
    }
    if (need > 0) {
        // The allocation around `ptr` must reach `need` bytes past it: a
        // descriptor larger than its memory would make the kernel read or
        // write outside the allocation.  Where the runtime reports no
        // allocation range for the pointer, the extent cannot be checked.
        hipDeviceptr_t lo = nullptr;
        size_t size = 0;
        const hipError_t re = hipMemGetAddressRange(&lo, &size, const_cast<void *>(ptr));
        if (re != hipSuccess) {
            (void)hipGetLastError();
        } else {
            const uintptr_t a = reinterpret_cast<uintptr_t>(lo), p = reinterpret_cast<uintptr_t>(ptr);
            const uintptr_t b = a + size;
            if (p < a || p >= b || (uint64_t)(b - p) < (uint64_t)need)
                return fail(KVX_ERR_RANGE,
                            "%s (%p) needs %lld bytes, but its allocation [%p, +%zu) ends %lld "
                            "bytes after it",
                            name, ptr, (long long)need, lo, size,
                            (long long)(p < b && p >= a ? (int64_t)(b - p) : 0));
        }
    }
    *dev_ptr = dev_mem ? const_cast<void *>(ptr) : attr.devicePointer;
    if (is_host) *is_host = !dev_mem;
    return KVX_OK;
}

// Byte strides of (layer, page, kv, slot, head) for a pool layout, with the
// base moved to (layer0, kv0, head0) of the range the call copies; `heads`
// is how many heads it copies.
kvx::Side pool_side(const kvx_pool *p, void *base, const int32_t *pt, int64_t pt_len,
                    int32_t layer0, int32_t kv0, int32_t head0, int32_t heads) {
    const int64_t row = (int64_t)p->head_dim * p->elem_bytes;
    const int64_t L = p->num_layers, N = p->num_pages, C = p->num_kv, T = p->page_tokens,
                  H = p->num_heads;
    kvx::Side s{};
    const bool token_major = p->layout == KVX_LPCTHD || p->layout == KVX_PLCTHD;
    if (token_major) {
        s.s_h = row;
        s.s_t = H * row;
    } else {
        s.s_t = row;
        s.s_h = T * row;
    }
    s.s_c = T * H * row;
    if (p->layout == KVX_LPCTHD || p->layout == KVX_LPCHTD) {
        s.s_p = C * s.s_c;
        s.s_l = N * s.s_p;
    } else {
        s.s_l = C * s.s_c;
        s.s_p = L * s.s_l;
    }
    s.base = static_cast<char *>(base) + layer0 * s.s_l + kv0 * s.s_c + head0 * s.s_h;
    s.pt = pt;
    s.pt_len = pt_len;
    s.T = p->page_tokens;
    s.N = p->num_pages;
    // The copied heads of consecutive slots form one run when each slot's
    // copied rows are adjacent and slots follow each other without a gap.
    s.tok_contig = s.s_t == heads * row && (heads == 1 || s.s_h == row);
    s.cap_bytes = 0;
    return s;
}

kvx::Side buf_side(const kvx_buf *b, void *base) {
    kvx::Side s{};
    s.base = static_cast<char *>(base);
    s.tok_contig = 1;
    s.T = 1;
    s.N = 0;
    s.cap_bytes = b->capacity_elems * b->elem_bytes;
    return s;
}

// Host-only checks of a pool descriptor (no HIP call).
int check_pool(const kvx_pool *p, const char *name, Shape &s) {
    int st = pool_shape(p, name, s);
    if (st) return st;
    if (!p->base) return fail(KVX_ERR_NULL, "%s: base is NULL", name);
    if (!aligned16(p->base)) return fail(KVX_ERR_ALIGN, "%s: base %p is not 16-byte aligned", name, p->base);
    if (pool_bytes(p) < 0) return fail(KVX_ERR_RANGE, "%s: pool size exceeds 2^63 bytes", name);
    return KVX_OK;
}

// Host-only checks of a buffer descriptor.
int check_buf(const kvx_buf *b, const char *name, Shape &s) {
    if (!b) return fail(KVX_ERR_NULL, "%s: buffer descriptor is NULL", name);
    s = Shape{b->num_layers, b->num_kv, b->num_heads, b->head_dim, b->elem_bytes};
    int st = check_shape(name, s);
    if (st) return st;
    if (b->reserved != 0) return fail(KVX_ERR_RANGE, "%s: reserved field must be 0", name);
    // An empty buffer may have no memory at all: no record can then address it.
    if (!b->base && b->capacity_elems != 0) return fail(KVX_ERR_NULL, "%s: base is NULL", name);
    if (!aligned16(b->base)) return fail(KVX_ERR_ALIGN, "%s: base %p is not 16-byte aligned", name, b->base);
    if (b->capacity_elems < 0 || mul_checked(b->capacity_elems, b->elem_bytes) < 0)
        return fail(KVX_ERR_RANGE, "%s: capacity_elems out of range", name);
    return KVX_OK;
}

// Host-only checks of a page table.
int check_table(const int32_t *pt, int64_t len, const char *name) {
    if (len < 0 || len > INT64_MAX / 4) return fail(KVX_ERR_RANGE, "%s: length %lld out of range", name,
                                                    (long long)len);
    if (len > 0 && !pt) return fail(KVX_ERR_NULL, "%s is NULL but has %lld entries", name, (long long)len);
    if ((reinterpret_cast<uintptr_t>(pt) & 3u) != 0) return fail(KVX_ERR_ALIGN, "%s is not 4-byte aligned", name);
    return KVX_OK;
}

// Host-only checks of the record array and the error word.
int check_common(const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err) {
    if (n_reqs < 0 || n_reqs > KVX_MAX_REQS)
        return fail(KVX_ERR_RANGE, "n_reqs %d outside [0, %d]", n_reqs, KVX_MAX_REQS);
    if (n_reqs > 0 && !reqs) return fail(KVX_ERR_NULL, "reqs is NULL");
    if ((reinterpret_cast<uintptr_t>(reqs) & 7u) != 0) return fail(KVX_ERR_ALIGN, "reqs is not 8-byte aligned");
    if ((reinterpret_cast<uintptr_t>(dev_err) & 3u) != 0)
        return fail(KVX_ERR_ALIGN, "dev_err is not 4-byte aligned");
    return KVX_OK;
}

// Device views of every pointer a launch uses.
struct Views {
    void *src = nullptr, *dst = nullptr;
    bool dst_host = false;
    const int32_t *src_pt = nullptr, *dst_pt = nullptr;
    const kvx_req *reqs = nullptr;
    uint32_t *err = nullptr;
};

int view_all(const void *src, int64_t src_bytes, const void *dst, int64_t dst_bytes,
             const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt, int64_t dst_pt_len,
             const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err, Views &v) {
    int st;
    void *d = nullptr;
    // A NULL base here is an empty buffer (pools are never NULL): nothing to view.
    if (src && (st = device_view(src, src_bytes, "src base", &v.src))) return st;
    if (dst && (st = device_view(dst, dst_bytes, "dst base", &v.dst, &v.dst_host))) return st;
    if (src_pt_len > 0) {
        if ((st = device_view(src_pt, src_pt_len * 4, "src_pt", &d))) return st;
        v.src_pt = static_cast<const int32_t *>(d);
    }
    if (dst_pt_len > 0) {
        if ((st = device_view(dst_pt, dst_pt_len * 4, "dst_pt", &d))) return st;
        v.dst_pt = static_cast<const int32_t *>(d);
    }
    if ((st = device_view(reqs, (int64_t)n_reqs * (int64_t)sizeof(kvx_req), "reqs", &d))) return st;
    v.reqs = static_cast<const kvx_req *>(d);
    if (dev_err) {
        // Bits are OR-ed in with device atomics, which pinned host memory
        // does not support on every platform: the word lives in device memory.
        if ((st = device_view(dev_err, 4, "dev_err", &d, nullptr, /*device_only=*/true))) return st;
        v.err = static_cast<uint32_t *>(d);
    }
    return KVX_OK;
}

// `s` gives the layers, kv components and heads the call copies.
void finish_params(kvx::Params &P, const Shape &s, const Views &v, int32_t n_reqs) {
    P.reqs = v.reqs;
    P.err = v.err;
    P.n_reqs = n_reqs;
    P.L = s.L;
    P.C = s.C;
    P.H = s.H;
    P.row_bytes = s.D * s.e;
    P.vpr = P.row_bytes / 16;
    P.elem_bytes = s.e;
    P.flat = P.src.tok_contig && P.dst.tok_contig;
    P.dst_host = v.dst_host;
    const kvx::Side &os = P.op == kvx::OP_GATHER ? P.dst : P.src;
    P.fd_vpr = kvx::make_fastdiv((uint32_t)P.vpr);
    P.fd_H = kvx::make_fastdiv((uint32_t)P.H);
    P.fd_To = kvx::make_fastdiv((uint32_t)os.T);
    P.fd_Tt = kvx::make_fastdiv((uint32_t)(P.op == kvx::OP_GATHER ? P.src : P.dst).T);
}

int enqueue(const kvx::Params &P, void *stream) {
    int e = kvx::launch(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail(KVX_ERR_HIP, "kernel launch failed: %s", hipGetErrorString((hipError_t)e));
    g_last_launch = P.sweep ? KVX_LAUNCH_SWEEP : KVX_LAUNCH_GRID;
    return KVX_OK;
}

// A slice's ranges must lie inside both pools; rows must have the same
// width on both sides.
int check_slice(const kvx_slice &sl, const Shape &s, const Shape &d) {
    if (s.D != d.D || s.e != d.e)
        return fail(KVX_ERR_SHAPE, "head_dim/elem_bytes differ: (%d, %d) vs (%d, %d)", s.D, s.e,
                    d.D, d.e);
    if (sl.reserved != 0) return fail(KVX_ERR_RANGE, "slice: reserved field must be 0");
    const struct {
        const char *what;
        int32_t s0, d0, n, smax, dmax;
    } r[3] = {{"layer", sl.src_layer0, sl.dst_layer0, sl.num_layers, s.L, d.L},
              {"kv", sl.src_kv0, sl.dst_kv0, sl.num_kv, s.C, d.C},
              {"head", sl.src_head0, sl.dst_head0, sl.num_heads, s.H, d.H}};
    for (const auto &x : r) {
        if (x.n < 0 || x.s0 < 0 || x.d0 < 0 || (int64_t)x.s0 + x.n > x.smax ||
            (int64_t)x.d0 + x.n > x.dmax)
            return fail(KVX_ERR_RANGE,
                        "slice %s range: src [%d, %lld) of %d, dst [%d, %lld) of %d", x.what, x.s0,
                        (long long)x.s0 + x.n, x.smax, x.d0, (long long)x.d0 + x.n, x.dmax);
    }
    return KVX_OK;
}

// Pool -> pool; slice == NULL copies everything between equal shapes.  With
// group > 0 the layer range is moved in groups of `group` layers, one launch
// each, and events[g] is recorded on the stream after group g.
// A planned transfer whose shape the sweep kernel serves well gets its
// launch: at least KVX_SWEEP_MIN_BYTES copied per destination page and layer
// on average, page tables whose indices fit in int32, and a grid of at most
// KVX_SWEEP_MAX_BLOCKS workgroups per pass.  Otherwise, and for unplanned
// calls, the persistent grid.
void plan_sweep(kvx::Params &P, const void *plan, int64_t plan_pages, int64_t plan_tokens) {
    P.sweep = 0;
    if (!plan || plan_pages < 1 || plan_tokens < 1 || P.n_reqs < 1 || P.op != kvx::OP_TRANSFER) return;
    if (P.src.pt_len > INT32_MAX || P.dst.pt_len > INT32_MAX) return;
    // rows per head of a page's enumeration: a head-major destination takes
    // whole blocks of slots, aligned to the page, so any slot range of a page
    // covers at most its ceil(T / block) blocks
    constexpr int64_t SB = KVX_SWEEP_SLOT_BLOCK;
    const int64_t T = P.dst.T, rows_per_head = P.dst.tok_contig ? T : (T + SB - 1) / SB * SB;
    // average bytes copied per destination page and layer
    const int64_t token_bytes = (int64_t)P.C * P.H * P.row_bytes;
    if (plan_tokens > INT64_MAX / token_bytes || plan_tokens * token_bytes < KVX_SWEEP_MIN_BYTES * plan_pages)
        return;
    // pieces of 64 vectors per page: the vectors of the page's enumeration
    const int64_t tile_vecs = (int64_t)P.C * rows_per_head * P.H * P.vpr;
    // workgroups per page: KVX_SWEEP_PIECES pieces each
    const int64_t ppt = ((tile_vecs + 63) / 64 + KVX_SWEEP_PIECES - 1) / KVX_SWEEP_PIECES;
    const int64_t per_slot = (int64_t)P.L * ppt;         // workgroups per page slot
    if (per_slot > KVX_SWEEP_MAX_BLOCKS) return;
    // page slots per pass: the plan's pages in KVX_SWEEP_PASSES passes (fewer
    // for small pages), within the grid cap
    const int64_t passes = plan_tokens * token_bytes < KVX_SWEEP_SMALL_BYTES * plan_pages
                               ? KVX_SWEEP_PASSES_SMALL : KVX_SWEEP_PASSES;
    const int64_t want = (plan_pages + passes - 1) / passes;
    const int64_t slots = want < KVX_SWEEP_MAX_BLOCKS / per_slot ? want : KVX_SWEEP_MAX_BLOCKS / per_slot;
    P.sweep = 1;
    P.prefix = static_cast<const int64_t *>(plan);
    P.slots = reinterpret_cast<const kvx_plan_slot *>(P.prefix + P.n_reqs + 1);
    P.plan_pages = plan_pages;
    P.sweep_pages = (int32_t)slots;
    P.sweep_ppt = (uint32_t)ppt;
    P.fd_ppt = kvx::make_fastdiv((uint32_t)ppt);
    P.fd_sp = kvx::make_fastdiv((uint32_t)slots);
    P.fd_hv = kvx::make_fastdiv((uint32_t)(P.H * P.vpr));
}

#ifndef KVX_LAUNCH_CHOICE_DEFAULT
#define KVX_LAUNCH_CHOICE_DEFAULT KVX_CHOOSE_MEASURED
#endif

// Launch choice of a planned single-launch transfer that can sweep (the
// rules are in include/kvx.h, kvx_set_launch_choice).  Both launches write
// the same bytes.  Which one is faster depends on where the pools sit in
// physical memory: for MLA's 72 KiB pages the persistent grid ran 1-8%
// above the sweep in most fresh processes and 3-9% below it in the rest,
// while each process's own rate held within 0.3% once warm.  So the first
// calls on a pair of pools warm both launches, then time both, and later
// calls keep the faster.  The key is the pair of pools (and the slice), not
// the records: a serving loop moves other requests in every call.
struct TuneKey {
    int dev;
    const void *src, *dst;
    kvx_pool sp, dp;
    kvx_slice sl;
};

// After six untimed calls (the launches in turn), four timed calls in the
// order sweep, grid, grid, sweep.  The first calls on fresh pools run slow
// (the first by up to 30%, and short ones for a few milliseconds more, the
// sweep longer than the grid); the order of the timed calls makes a drift
// that remains weigh on both sums alike.
constexpr int kUntimed = 6;
constexpr int kTimed = 4;
constexpr int kTimedLaunch[kTimed] = {KVX_LAUNCH_SWEEP, KVX_LAUNCH_GRID, KVX_LAUNCH_GRID,
                                      KVX_LAUNCH_SWEEP};

struct Tune {
    TuneKey key;
    int calls;                 // calls seen before the decision
    int choice;                // KVX_LAUNCH_SWEEP or KVX_LAUNCH_GRID once decided, else 0
    hipEvent_t ev[2 * kTimed]; // start and end of each timed call
    int64_t tokens[kTimed];    // tokens each timed call moved (calls may move different amounts)
    uint64_t used;             // recency, for dropping the least recently used key
};

constexpr size_t kMaxTunes = 64;
std::mutex g_tune_mu;
std::vector<Tune> g_tunes;   // never destroyed: events are not released at exit
uint64_t g_tune_clock = 0;
std::atomic<int> g_choice_mode{KVX_LAUNCH_CHOICE_DEFAULT};

void drop_events(Tune &t) {
    for (hipEvent_t &e : t.ev)
        if (e) {
            (void)hipEventDestroy(e);
            e = nullptr;
        }
}

// Decides t once every timed call has completed (false while one is
// pending): the launch that moved more tokens per millisecond over its two
// timed calls.
bool decide(Tune &t) {
    double ms_sum[3] = {0.0, 0.0, 0.0}, tok_sum[3] = {0.0, 0.0, 0.0};   // by launch kind
    bool ok = true;
    for (int k = 0; k < kTimed && ok; ++k) {
        const hipError_t q = hipEventQuery(t.ev[2 * k + 1]);
        if (q == hipErrorNotReady) return false;
        float ms = 0.f;
        ok = q == hipSuccess && hipEventElapsedTime(&ms, t.ev[2 * k], t.ev[2 * k + 1]) == hipSuccess &&
             ms > 0.f;
        ms_sum[kTimedLaunch[k]] += ms;
        tok_sum[kTimedLaunch[k]] += (double)t.tokens[k];
    }
    // grid faster: tok_g / ms_g > tok_s / ms_s
    t.choice = ok && tok_sum[KVX_LAUNCH_GRID] * ms_sum[KVX_LAUNCH_SWEEP] >
                         tok_sum[KVX_LAUNCH_SWEEP] * ms_sum[KVX_LAUNCH_GRID]
                   ? KVX_LAUNCH_GRID : KVX_LAUNCH_SWEEP;
    drop_events(t);
    return true;
}

// The launch for this call (KVX_LAUNCH_SWEEP or KVX_LAUNCH_GRID) and, when
// the call is timed, the events to record around it (else null); tokens is
// what the call moves.  Called with g_tune_mu held.
int pick_launch(const TuneKey &key, int64_t tokens, hipStream_t stream, hipEvent_t *t0,
                hipEvent_t *t1) {
    *t0 = *t1 = nullptr;
    if (g_choice_mode == KVX_CHOOSE_SWEEP) return KVX_LAUNCH_SWEEP;
    if (g_choice_mode == KVX_CHOOSE_GRID) return KVX_LAUNCH_GRID;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const bool capturing = hipStreamIsCapturing(stream, &cs) != hipSuccess ||
                           cs != hipStreamCaptureStatusNone;
    Tune *t = nullptr;
    for (Tune &x : g_tunes)
        if (std::memcmp(&x.key, &key, sizeof key) == 0) t = &x;
    if (!t) {
        if (capturing) return KVX_LAUNCH_SWEEP;
        if (g_tunes.size() == kMaxTunes) {
            auto old = std::min_element(g_tunes.begin(), g_tunes.end(),
                                        [](const Tune &a, const Tune &b) { return a.used < b.used; });
            drop_events(*old);
            g_tunes.erase(old);
        }
        g_tunes.push_back(Tune{});
        t = &g_tunes.back();
        std::memcpy(&t->key, &key, sizeof key);   // padding included: keys compare with memcmp
    }
    t->used = ++g_tune_clock;
    if (t->choice) return t->choice;
    if (capturing) return KVX_LAUNCH_SWEEP;
    const int k = t->calls - kUntimed;          // index of this call among the timed ones
    if (k >= kTimed) return decide(*t) ? t->choice : KVX_LAUNCH_SWEEP;
    ++t->calls;
    if (k < 0) return (k + kUntimed) % 2 ? KVX_LAUNCH_GRID : KVX_LAUNCH_SWEEP;   // untimed
    if (k == 0)
        for (hipEvent_t &e : t->ev)
            if (hipEventCreate(&e) != hipSuccess) {
                e = nullptr;
                drop_events(*t);
                t->choice = KVX_LAUNCH_SWEEP;
                return t->choice;
            }
    *t0 = t->ev[2 * k];
    *t1 = t->ev[2 * k + 1];
    t->tokens[k] = tokens;
    return kTimedLaunch[k];
}

// Enqueue P (one launch of a transfer that plan_sweep may have set to sweep)
// with the launch pick_launch gives.  A timed call records its events and
// launches with the lock still held, so that no other call of the key
// queries or destroys the events before they are recorded.
int enqueue_chosen(kvx::Params &P, const TuneKey &key, int64_t tokens, void *stream) {
    if (!P.sweep) return enqueue(P, stream);
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    hipEvent_t t0, t1;
    std::unique_lock<std::mutex> lock(g_tune_mu);
    P.sweep = pick_launch(key, tokens, hs, &t0, &t1) == KVX_LAUNCH_SWEEP;
    if (!t0) {
        lock.unlock();
        return enqueue(P, stream);
    }
    if (hipEventRecord(t0, hs) != hipSuccess) t1 = nullptr;
    const int st = enqueue(P, stream);
    if (st == KVX_OK && t1) (void)hipEventRecord(t1, hs);
    return st;
}

int transfer_impl(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                  const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt,
                  int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err,
                  void *stream, int32_t group = 0, void *const *events = nullptr,
                  int32_t n_events = 0, const void *plan = nullptr, int64_t plan_pages = -1,
                  int64_t plan_tokens = -1) {
    g_last_launch = KVX_LAUNCH_NONE;
    Shape ss, ds;
    int st;
    if ((st = check_pool(src, "src", ss))) return st;
    if ((st = check_pool(dst, "dst", ds))) return st;
    kvx_slice sl;
    if (slice) {
        sl = *slice;
        if ((st = check_slice(sl, ss, ds))) return st;
    } else {
        if ((st = same_shape(ss, ds))) return st;
        sl = kvx_slice{0, 0, ss.L, 0, 0, ss.C, 0, 0, ss.H, 0};
    }
    if ((st = check_common(reqs, n_reqs, dev_err))) return st;
    if ((st = check_table(src_pt, src_pt_len, "src_pt"))) return st;
    if ((st = check_table(dst_pt, dst_pt_len, "dst_pt"))) return st;
    int32_t groups = 1;
    if (group > 0) {
        groups = sl.num_layers == 0 ? 0 : (sl.num_layers + group - 1) / group;
        if (n_events < groups)
            return fail(KVX_ERR_RANGE, "%d layer groups need %d events, got %d", groups, groups,
                        n_events);
        if (groups > 0 && !events) return fail(KVX_ERR_NULL, "events is NULL");
        for (int32_t g = 0; g < groups; ++g)
            if (!events[g]) return fail(KVX_ERR_NULL, "events[%d] is NULL", g);
    }
    const bool empty = n_reqs == 0 || sl.num_layers == 0 || sl.num_kv == 0 || sl.num_heads == 0;
    Views v;
    if (!empty && (st = view_all(src->base, pool_bytes(src), dst->base, pool_bytes(dst), src_pt,
                                 src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs, dev_err, v)))
        return st;
    if (!empty && plan) {
        void *d = nullptr;
        if ((st = device_view(plan, KVX_PLAN_BYTES(n_reqs, plan_pages), "plan", &d))) return st;
        plan = d;
    }
    const hipStream_t hs = static_cast<hipStream_t>(stream);
    for (int32_t g = 0; g < groups; ++g) {
        if (!empty) {
            const int32_t l0 = group > 0 ? g * group : 0;
            const int32_t nl = group > 0 ? std::min(group, sl.num_layers - l0) : sl.num_layers;
            kvx::Params P{};
            P.op = kvx::OP_TRANSFER;
            P.src = pool_side(src, v.src, v.src_pt, src_pt_len, sl.src_layer0 + l0, sl.src_kv0,
                              sl.src_head0, sl.num_heads);
            P.dst = pool_side(dst, v.dst, v.dst_pt, dst_pt_len, sl.dst_layer0 + l0, sl.dst_kv0,
                              sl.dst_head0, sl.num_heads);
            finish_params(P, Shape{nl, sl.num_kv, sl.num_heads, ss.D, ss.e}, v, n_reqs);
            plan_sweep(P, plan, plan_pages, plan_tokens);
            if (group > 0) {
                if (g_choice_mode == KVX_CHOOSE_GRID) P.sweep = 0;
                st = enqueue(P, stream);
            } else {
                TuneKey key;
                std::memset(&key, 0, sizeof key);
                if (hipGetDevice(&key.dev) != hipSuccess) key.dev = -1;
                key.src = src->base;
                key.dst = dst->base;
                key.sp = *src;
                key.dp = *dst;
                key.sl = sl;
                st = enqueue_chosen(P, key, plan_tokens, stream);
            }
            if (st) return st;
        }
        if (group > 0) {
            const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(events[g]), hs);
            if (e != hipSuccess)
                return fail(KVX_ERR_HIP, "recording the event of layer group %d failed: %s", g,
                            hipGetErrorString(e));
        }
    }
    return KVX_OK;
}

// A buffer that holds exactly a slice of a pool: the pool's range inside the
// pool, the buffer-side offsets zero and the buffer's layer, kv and head
// counts equal to the slice's.  `pool_is_src` picks which offsets are the
// pool's (source fields for a gather, destination fields for a scatter).
int check_buffer_slice(const kvx_slice &sl, const Shape &pool, const Shape &buf, bool pool_is_src) {
    if (pool.D != buf.D || pool.e != buf.e)
        return fail(KVX_ERR_SHAPE, "head_dim/elem_bytes differ: (%d, %d) vs (%d, %d)", pool.D, pool.e,
                    buf.D, buf.e);
    if (sl.reserved != 0) return fail(KVX_ERR_RANGE, "slice: reserved field must be 0");
    const struct {
        const char *what;
        int32_t p0, b0, n, pmax, bn;
    } r[3] = {{"layer", pool_is_src ? sl.src_layer0 : sl.dst_layer0,
               pool_is_src ? sl.dst_layer0 : sl.src_layer0, sl.num_layers, pool.L, buf.L},
              {"kv", pool_is_src ? sl.src_kv0 : sl.dst_kv0, pool_is_src ? sl.dst_kv0 : sl.src_kv0,
               sl.num_kv, pool.C, buf.C},
              {"head", pool_is_src ? sl.src_head0 : sl.dst_head0,
               pool_is_src ? sl.dst_head0 : sl.src_head0, sl.num_heads, pool.H, buf.H}};
    for (const auto &x : r) {
        if (x.n < 0 || x.p0 < 0 || (int64_t)x.p0 + x.n > x.pmax)
            return fail(KVX_ERR_RANGE, "slice %s range [%d, %lld) outside the pool's %d", x.what, x.p0,
                        (long long)x.p0 + x.n, x.pmax);
        if (x.b0 != 0)
            return fail(KVX_ERR_RANGE, "slice %s offset on the buffer side must be 0 (got %d)", x.what,
                        x.b0);
        if (x.n != x.bn)
            return fail(KVX_ERR_SHAPE, "the buffer holds %d %s(s), the slice %d", x.bn, x.what, x.n);
    }
    return KVX_OK;
}

// Pool <-> flat buffer.  `op` is OP_GATHER (pool -> buffer) or OP_SCATTER
// (buffer -> pool); slice == NULL moves everything between equal shapes.
int buffer_impl(int op, const kvx_pool *pool, const kvx_buf *buf, const kvx_slice *slice,
                const int32_t *pt, int64_t pt_len, const kvx_req *reqs, int32_t n_reqs,
                uint32_t *dev_err, void *stream) {
    g_last_launch = KVX_LAUNCH_NONE;
    const bool gather = op == kvx::OP_GATHER;
    const char *pname = gather ? "src" : "dst", *bname = gather ? "dst" : "src";
    const char *tname = gather ? "src_pt" : "dst_pt";
    Shape ps, bs;
    int st;
    if (gather) {
        if ((st = check_pool(pool, pname, ps))) return st;
        if ((st = check_buf(buf, bname, bs))) return st;
    } else {
        if ((st = check_buf(buf, bname, bs))) return st;
        if ((st = check_pool(pool, pname, ps))) return st;
    }
    kvx_slice sl;
    if (slice) {
        sl = *slice;
        if ((st = check_buffer_slice(sl, ps, bs, gather))) return st;
    } else {
        if ((st = same_shape(ps, bs))) return st;
        sl = kvx_slice{0, 0, ps.L, 0, 0, ps.C, 0, 0, ps.H, 0};
    }
    if ((st = check_common(reqs, n_reqs, dev_err))) return st;
    if ((st = check_table(pt, pt_len, tname))) return st;
    if (n_reqs == 0) return KVX_OK;
    Views v;
    const int64_t buf_bytes = buf->capacity_elems * buf->elem_bytes;
    if (gather)
        st = view_all(pool->base, pool_bytes(pool), buf->base, buf_bytes, pt, pt_len, nullptr, 0,
                      reqs, n_reqs, dev_err, v);
    else
        st = view_all(buf->base, buf_bytes, pool->base, pool_bytes(pool), nullptr, 0, pt, pt_len,
                      reqs, n_reqs, dev_err, v);
    if (st) return st;
    const int32_t l0 = gather ? sl.src_layer0 : sl.dst_layer0;
    const int32_t c0 = gather ? sl.src_kv0 : sl.dst_kv0;
    const int32_t h0 = gather ? sl.src_head0 : sl.dst_head0;
    kvx::Params P{};
    P.op = op;
    if (gather) {
        P.src = pool_side(pool, v.src, v.src_pt, pt_len, l0, c0, h0, sl.num_heads);
        P.dst = buf_side(buf, v.dst);
    } else {
        P.src = buf_side(buf, v.src);
        P.dst = pool_side(pool, v.dst, v.dst_pt, pt_len, l0, c0, h0, sl.num_heads);
    }
    finish_params(P, Shape{sl.num_layers, sl.num_kv, sl.num_heads, ps.D, ps.e}, v, n_reqs);
    return enqueue(P, stream);
}

}  // namespace

extern "C" {

int kvx_transfer(const kvx_pool *src, const kvx_pool *dst, const int32_t *src_pt, int64_t src_pt_len,
                 const int32_t *dst_pt, int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs,
                 uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    return transfer_impl(src, dst, nullptr, src_pt, src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs,
                         dev_err, stream);
}

int kvx_transfer_slice(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                       const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt,
                       int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err,
                       void *stream) {
    g_last_error.clear();
    if (!slice) return fail(KVX_ERR_NULL, "slice is NULL");
    return transfer_impl(src, dst, slice, src_pt, src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs,
                         dev_err, stream);
}

int kvx_gather(const kvx_pool *src, const kvx_buf *dst, const int32_t *src_pt, int64_t src_pt_len,
               const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    return buffer_impl(kvx::OP_GATHER, src, dst, nullptr, src_pt, src_pt_len, reqs, n_reqs, dev_err,
                       stream);
}

int kvx_scatter(const kvx_buf *src, const kvx_pool *dst, const int32_t *dst_pt, int64_t dst_pt_len,
                const kvx_req *reqs, int32_t n_reqs, uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    return buffer_impl(kvx::OP_SCATTER, dst, src, nullptr, dst_pt, dst_pt_len, reqs, n_reqs, dev_err,
                       stream);
}

int kvx_gather_slice(const kvx_pool *src, const kvx_buf *dst, const kvx_slice *slice,
                     const int32_t *src_pt, int64_t src_pt_len, const kvx_req *reqs, int32_t n_reqs,
                     uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    if (!slice) return fail(KVX_ERR_NULL, "slice is NULL");
    return buffer_impl(kvx::OP_GATHER, src, dst, slice, src_pt, src_pt_len, reqs, n_reqs, dev_err,
                       stream);
}

int kvx_scatter_slice(const kvx_buf *src, const kvx_pool *dst, const kvx_slice *slice,
                      const int32_t *dst_pt, int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs,
                      uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    if (!slice) return fail(KVX_ERR_NULL, "slice is NULL");
    return buffer_impl(kvx::OP_SCATTER, dst, src, slice, dst_pt, dst_pt_len, reqs, n_reqs, dev_err,
                       stream);
}

int kvx_transfer_planned(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                         const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt,
                         int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs, const void *plan,
                         int64_t plan_pages, int64_t plan_tokens, uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    // the prefix holds n_reqs + 1 words and every record has fewer than 2^31 pages
    if (plan_pages < 0 || plan_tokens < 0 || plan_pages > (int64_t)KVX_MAX_REQS * INT32_MAX)
        return fail(KVX_ERR_RANGE, "plan_pages and plan_tokens must be >= 0 (got %lld, %lld)",
                    (long long)plan_pages, (long long)plan_tokens);
    if (n_reqs > 0 && !plan) return fail(KVX_ERR_NULL, "plan is NULL");
    if ((reinterpret_cast<uintptr_t>(plan) & 7u) != 0) return fail(KVX_ERR_ALIGN, "plan is not 8-byte aligned");
    return transfer_impl(src, dst, slice, src_pt, src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs,
                         dev_err, stream, 0, nullptr, 0, plan, plan_pages, plan_tokens);
}

int kvx_transfer_layered_planned(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                                 const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt,
                                 int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs,
                                 int32_t layers_per_group, void *const *events, int32_t n_events,
                                 const void *plan, int64_t plan_pages, int64_t plan_tokens,
                                 uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    if (layers_per_group < 1)
        return fail(KVX_ERR_RANGE, "layers_per_group must be >= 1 (got %d)", layers_per_group);
    if (plan_pages < 0 || plan_tokens < 0 || plan_pages > (int64_t)KVX_MAX_REQS * INT32_MAX)
        return fail(KVX_ERR_RANGE, "plan_pages and plan_tokens must be >= 0 (got %lld, %lld)",
                    (long long)plan_pages, (long long)plan_tokens);
    if (n_reqs > 0 && !plan) return fail(KVX_ERR_NULL, "plan is NULL");
    if ((reinterpret_cast<uintptr_t>(plan) & 7u) != 0) return fail(KVX_ERR_ALIGN, "plan is not 8-byte aligned");
    return transfer_impl(src, dst, slice, src_pt, src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs,
                         dev_err, stream, layers_per_group, events, n_events, plan, plan_pages,
                         plan_tokens);
}

int64_t kvx_plan_pages(const kvx_req *host_reqs, int32_t n_reqs, int32_t page_tokens, int32_t side,
                       int64_t *prefix, int64_t *tokens) {
    g_last_error.clear();
    if (n_reqs < 0 || n_reqs > KVX_MAX_REQS || (n_reqs > 0 && !host_reqs) || page_tokens < 1 ||
        (side != 0 && side != 1)) {
        fail(KVX_ERR_RANGE, "kvx_plan_pages: bad arguments");
        return -1;
    }
    int64_t pages = 0, n_tok = 0;
    for (int32_t r = 0; r < n_reqs; ++r) {
        if (prefix) prefix[r] = pages;
        const kvx_req &R = host_reqs[r];
        // a malformed record (the kvx_req rules that do not depend on a buffer) counts 0
        const int64_t s0 = R.src_start, d0 = R.dst_start, n = R.n_tokens;
        if (n <= 0 || s0 < 0 || d0 < 0 || R.reserved != 0 || s0 + n > INT32_MAX || d0 + n > INT32_MAX)
            continue;
        const int64_t start = side ? d0 : s0;
        pages += (start + n - 1) / page_tokens - start / page_tokens + 1;
        n_tok += n;
    }
    if (prefix) prefix[n_reqs] = pages;
    if (tokens) *tokens = n_tok;
    return pages;
}

namespace {
int32_t clamp_i32(int64_t x) { return x < INT32_MIN ? INT32_MIN : x > INT32_MAX ? INT32_MAX : (int32_t)x; }
}  // namespace

int kvx_plan_fill(const kvx_req *host_reqs, int32_t n_reqs, int32_t src_page_tokens,
                  int32_t dst_page_tokens, int64_t plan_pages, void *plan) {
    g_last_error.clear();
    if (n_reqs < 0 || n_reqs > KVX_MAX_REQS || src_page_tokens < 1 || dst_page_tokens < 1 || plan_pages < 0)
        return fail(KVX_ERR_RANGE, "kvx_plan_fill: bad arguments");
    if ((n_reqs > 0 && !host_reqs) || !plan) return fail(KVX_ERR_NULL, "kvx_plan_fill: NULL pointer");
    if ((reinterpret_cast<uintptr_t>(plan) & 7u) != 0) return fail(KVX_ERR_ALIGN, "plan is not 8-byte aligned");
    int64_t *prefix = static_cast<int64_t *>(plan);
    const int64_t total = kvx_plan_pages(host_reqs, n_reqs, dst_page_tokens, 1, prefix, nullptr);
    if (total != plan_pages)
        return fail(KVX_ERR_RANGE, "plan_pages %lld differs from the records' %lld pages",
                    (long long)plan_pages, (long long)total);
    kvx_plan_slot *slot = reinterpret_cast<kvx_plan_slot *>(prefix + n_reqs + 1);
    const int64_t Td = dst_page_tokens, Ts = src_page_tokens;
    for (int32_t r = 0; r < n_reqs; ++r) {
        const kvx_req &R = host_reqs[r];
        const int64_t pages = prefix[r + 1] - prefix[r];
        const int64_t d0 = R.dst_start, s0 = R.src_start, end = d0 + R.n_tokens;
        for (int64_t jj = 0; jj < pages; ++jj, ++slot) {
            const int64_t j = d0 / Td + jj, page_lo = j * Td;
            const int64_t qa = page_lo > d0 ? page_lo : d0;
            const int64_t qb = page_lo + Td < end ? page_lo + Td : end;
            const int64_t pos = qa - d0 + s0;              // source position of the first token
            *slot = kvx_plan_slot{clamp_i32(R.dst_pt_off + j), clamp_i32(R.src_pt_off + pos / Ts),
                                  (int32_t)(qa - page_lo), (int32_t)(qb - qa), (int32_t)(pos % Ts), r,
                                  {0, 0}};
        }
    }
    return KVX_OK;
}

int kvx_transfer_layered(const kvx_pool *src, const kvx_pool *dst, const kvx_slice *slice,
                         const int32_t *src_pt, int64_t src_pt_len, const int32_t *dst_pt,
                         int64_t dst_pt_len, const kvx_req *reqs, int32_t n_reqs,
                         int32_t layers_per_group, void *const *events, int32_t n_events,
                         uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    if (layers_per_group < 1)
        return fail(KVX_ERR_RANGE, "layers_per_group must be >= 1 (got %d)", layers_per_group);
    return transfer_impl(src, dst, slice, src_pt, src_pt_len, dst_pt, dst_pt_len, reqs, n_reqs,
                         dev_err, stream, layers_per_group, events, n_events);
}

int kvx_page_hashes(const void *payload, int64_t payload_positions, int32_t rec_bytes,
                    int32_t page_tokens, const kvx_hash_req *reqs, int32_t n_reqs, uint64_t *out,
                    int64_t out_len, uint32_t *dev_err, void *stream) {
    g_last_error.clear();
    if (rec_bytes < 4 || rec_bytes % 4 != 0)
        return fail(KVX_ERR_SHAPE, "rec_bytes must be a positive multiple of 4 (got %d)", rec_bytes);
    if (page_tokens < 1 || page_tokens > KVX_MAX_PAGE_TOKENS)
        return fail(KVX_ERR_SHAPE, "page_tokens %d outside [1, %d]", page_tokens, KVX_MAX_PAGE_TOKENS);
    if (payload_positions < 0 || out_len < 0 || out_len > INT64_MAX / 8)
        return fail(KVX_ERR_RANGE, "payload_positions and out_len must be >= 0 (and out_len < 2^60)");
    if (mul_checked(payload_positions, rec_bytes) < 0)
        return fail(KVX_ERR_RANGE, "payload size exceeds 2^63 bytes");
    if (n_reqs < 0 || n_reqs > KVX_MAX_REQS)
        return fail(KVX_ERR_RANGE, "n_reqs %d outside [0, %d]", n_reqs, KVX_MAX_REQS);
    if (n_reqs > 0 && !reqs) return fail(KVX_ERR_NULL, "reqs is NULL");
    if (payload_positions > 0 && !payload) return fail(KVX_ERR_NULL, "payload is NULL");
    if (out_len > 0 && !out) return fail(KVX_ERR_NULL, "out is NULL");
    if ((reinterpret_cast<uintptr_t>(payload) & 3u) != 0)
        return fail(KVX_ERR_ALIGN, "payload is not 4-byte aligned");
    if ((reinterpret_cast<uintptr_t>(out) & 7u) != 0 || (reinterpret_cast<uintptr_t>(reqs) & 7u) != 0)
        return fail(KVX_ERR_ALIGN, "out and reqs must be 8-byte aligned");
    if (!dev_err)
        return fail(KVX_ERR_NULL, "dev_err is required: it is the only signal of an incomplete chain");
    if ((reinterpret_cast<uintptr_t>(dev_err) & 3u) != 0)
        return fail(KVX_ERR_ALIGN, "dev_err is not 4-byte aligned");
    if (n_reqs == 0) return KVX_OK;
    kvx::HashParams P{};
    void *d = nullptr;
    int st;
    if (payload_positions > 0) {
        if ((st = device_view(payload, payload_positions * rec_bytes, "payload", &d))) return st;
        P.payload = static_cast<const uint32_t *>(d);
    }
    if (out_len > 0) {
        if ((st = device_view(out, out_len * 8, "out", &d))) return st;
        P.out = static_cast<uint64_t *>(d);
    }
    if ((st = device_view(reqs, (int64_t)n_reqs * (int64_t)sizeof(kvx_hash_req), "reqs", &d)))
        return st;
    P.reqs = static_cast<const kvx_hash_req *>(d);
    if ((st = device_view(dev_err, 4, "dev_err", &d, nullptr, /*device_only=*/true))) return st;
    P.err = static_cast<uint32_t *>(d);
    P.payload_positions = payload_positions;
    P.rec_bytes = rec_bytes;
    P.T = page_tokens;
    P.n_reqs = n_reqs;
    P.out_len = out_len;
    const int e = kvx::launch_hash(P, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail(KVX_ERR_HIP, "hash kernel launch failed: %s", hipGetErrorString((hipError_t)e));
    return KVX_OK;
}

int64_t kvx_pool_bytes(const kvx_pool *pool) {
    Shape s;
    if (!pool || pool_shape(pool, "pool", s) != KVX_OK) return -1;
    return pool_bytes(pool);
}

const char *kvx_strerror(int status) {
    switch (status) {
    case KVX_OK: return "success";
    case KVX_ERR_NULL: return "a required pointer is NULL";
    case KVX_ERR_SHAPE: return "element shapes differ or a dimension is out of range";
    case KVX_ERR_ALIGN: return "a pointer or row size is not 16-byte aligned";
    case KVX_ERR_LAYOUT: return "unknown layout or num_kv not 1 or 2";
    case KVX_ERR_RANGE: return "a count, size or pointer is out of range";
    case KVX_ERR_HIP: return "the HIP runtime reported an error";
    default: return "unknown kvx status";
    }
}

const char *kvx_last_error(void) { return g_last_error.c_str(); }

int kvx_set_launch_choice(int mode) {
    g_last_error.clear();
    if (mode != KVX_CHOOSE_MEASURED && mode != KVX_CHOOSE_SWEEP && mode != KVX_CHOOSE_GRID)
        return fail(KVX_ERR_RANGE, "launch choice %d is not a KVX_CHOOSE_* mode", mode);
    std::lock_guard<std::mutex> lock(g_tune_mu);
    for (Tune &t : g_tunes) drop_events(t);
    g_tunes.clear();
    g_choice_mode = mode;
    return KVX_OK;
}

int kvx_launch_choice(void) { return g_choice_mode.load(); }

int kvx_last_launch(void) { return g_last_launch; }

int kvx_abi_version(void) { return KVX_ABI_VERSION; }

}  // extern "C"
