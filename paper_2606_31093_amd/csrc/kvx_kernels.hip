// kvx_kernels.hip -- the copy engine of libkvx: HIP kernels for gfx950.
//
// One kernel moves the rows named by a batch of request records from a
// source side to a destination side (Omni-Flow Sec. 4.1.1: layer x page x
// slice addressing; Sec. 4.1.2: conversion between the paged layout and the
// flat serialization; Sec. 5.2: slot -> page translation through a table).
// Nothing is computed on the data: every element moves as raw bytes inside
// 16-byte vectors, so the kernel is bound by HBM (or the host link when a
// side is pinned host memory).
//
// Work decomposition.  A tile is (request r, page j of the tiling side,
// layer l); the tiling side is the destination pool for transfer and
// scatter (each tile then writes one destination page of one layer, and no
// two tiles write the same bytes) and the source pool for gather.  A
// persistent grid of workgroups strides over the flat tile index.  Each
// workgroup reads the request records 256 at a time, one per thread, turns
// their tile counts into tile ranges with a scan in LDS and finds the record
// of each of its tiles by binary search, so no tile table or scratch memory
// is needed and thousands of small requests cost a few parallel loads per
// chunk rather than a chain of dependent ones.  A tile is copied by one
// worker: a wavefront when the launch copies contiguous runs (four small
// tiles in flight per workgroup), the whole workgroup when it resolves rows.
//
// Inside a tile the tiling side's rows are a fixed page of one layer.  The
// other side's rows come from one or more of its pages ("pieces"), whose ids
// each wavefront loads once into lanes 0..K-1 and broadcasts with a lane
// shuffle.  When both sides keep the rows of consecutive tokens adjacent
// (token-major layouts and the flat buffer) and the tile maps onto a single
// piece, a tile is C contiguous runs on both sides and the copy is a plain
// vector stream; otherwise each 16-byte vector resolves its row.

#include "kvx_internal.h"

#ifndef KVX_UNROLL_FLAT
#define KVX_UNROLL_FLAT 8
#endif
#ifndef KVX_UNROLL_ROWS
#define KVX_UNROLL_ROWS 4
#endif
#ifndef KVX_NT
#define KVX_NT 1   // streaming (non-temporal) loads and stores: nothing is re-read
#endif
#ifndef KVX_NT_LOAD
#define KVX_NT_LOAD KVX_NT
#endif
#ifndef KVX_NT_STORE
#define KVX_NT_STORE KVX_NT
#endif
#ifndef KVX_ROWS_BLOCKS_PER_CU
#define KVX_ROWS_BLOCKS_PER_CU 3  // grid of launches that resolve rows (measured best)
#endif
#ifndef KVX_BLOCKS_PER_CU
#define KVX_BLOCKS_PER_CU 0  // 0: as many as fit
#endif
#ifndef KVX_BLOCK
#define KVX_BLOCK 256
#endif
#ifndef KVX_FLAT_WAVE_TILES
#define KVX_FLAT_WAVE_TILES 1  // launches of contiguous runs: one tile per wavefront
#endif
#ifndef KVX_ROWS_WAVE_TILES
#define KVX_ROWS_WAVE_TILES 0  // launches that resolve rows: one tile per workgroup
#endif

namespace kvx {
namespace {

constexpr int kBlock = KVX_BLOCK;
constexpr int kWave = 64;
// A worker copies one tile at a time: a wavefront or the whole workgroup,
// NT threads (a template parameter below).
template <int NT>
__device__ __forceinline__ uint32_t worker_tid() { return threadIdx.x % NT; }

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4u ld16(const char *p) {
#if KVX_NT_LOAD
    return __builtin_nontemporal_load(reinterpret_cast<const v4u *>(p));
#else
    return *reinterpret_cast<const v4u *>(p);
#endif
}

// Stores into device memory stream past the caches; stores into pinned host
// memory (HOST) are ordinary, which measured faster over PCIe.
template <bool HOST>
__device__ __forceinline__ void st16(char *p, v4u v) {
#if KVX_NT_STORE
    if (!HOST) {
        __builtin_nontemporal_store(v, reinterpret_cast<v4u *>(p));
        return;
    }
#endif
    *reinterpret_cast<v4u *>(p) = v;
}

// A read of data the kernel never writes (the plan, the records, the page
// tables) through the constant address space: the compiler may then serve a
// uniform one from the scalar cache wherever it falls, also after stores.
template <class T>
__device__ __forceinline__ T cload(const T *ptr) {
    static_assert(sizeof(T) % 4 == 0, "whole 32-bit words");
    typedef const __attribute__((address_space(4))) uint32_t cword;
    const cword *q = (const cword *)(uintptr_t)ptr;
    uint32_t w[sizeof(T) / 4];
#pragma unroll
    for (unsigned i = 0; i < sizeof(T) / 4; ++i) w[i] = q[i];
    T out;
    __builtin_memcpy(&out, w, sizeof(T));
    return out;
}

__device__ __forceinline__ void report(const Params &p, uint32_t bits) {
    if (p.err) atomicOr(p.err, bits);
}

// A request as one tile walk sees it.
struct Req {
    int64_t t_pt_off, o_pt_off;  // table offsets of the tiling / other side
    int64_t blk;                 // buffer block offset in bytes
    int64_t tiles;               // tiles this request contributes
    int64_t pages;               // tiling-side pages it touches (tiles = pages * layers)
    int32_t t_start, o_start, n;
    int32_t j0;                  // first tiling-side page (logical)
};

__device__ __forceinline__ bool block_fits(const Side &b, int64_t off, int32_t n,
                                           int64_t token_bytes, int32_t e) {
    if (off < 0 || off > b.cap_bytes / e) return false;
    const int64_t start = off * e;
    return (start & 15) == 0 && start + (int64_t)n * token_bytes <= b.cap_bytes;
}

template <int OP>
__device__ __forceinline__ bool load_req(const Params &p, int32_t r, Req &q) {
    const kvx_req &R = p.reqs[r];
    const int64_t so = R.src_pt_off, dof = R.dst_pt_off, bo = R.buf_off;
    const int32_t s0 = R.src_start, d0 = R.dst_start, n = R.n_tokens;
    bool ok = n >= 0 && s0 >= 0 && d0 >= 0 && R.reserved == 0 &&
              (int64_t)s0 + n <= INT32_MAX && (int64_t)d0 + n <= INT32_MAX;
    const int64_t token_bytes = (int64_t)p.L * p.C * p.H * p.row_bytes;
    if (OP == OP_GATHER) ok = ok && d0 == 0 && block_fits(p.dst, bo, n, token_bytes, p.elem_bytes);
    if (OP == OP_SCATTER) ok = ok && s0 == 0 && block_fits(p.src, bo, n, token_bytes, p.elem_bytes);
    if (!ok) {
        q.tiles = 0;
        q.pages = 0;
        return false;
    }
    const bool tsrc = OP == OP_GATHER;
    q.t_pt_off = tsrc ? so : dof;
    q.o_pt_off = tsrc ? dof : so;
    q.t_start = tsrc ? s0 : d0;
    q.o_start = tsrc ? d0 : s0;
    q.n = n;
    q.blk = bo * p.elem_bytes;
    if (n == 0) {
        q.tiles = 0;
        q.pages = 0;
        q.j0 = 0;
        return true;
    }
    const int32_t j0 = (int32_t)fd_div(p.fd_Tt, (uint32_t)q.t_start);
    const int32_t j1 = (int32_t)fd_div(p.fd_Tt, (uint32_t)(q.t_start + n - 1));
    q.j0 = j0;
    q.pages = j1 - j0 + 1;
    q.tiles = q.pages * p.L;
    return true;
}

// Plain vector stream over C runs of R vectors each, by a worker of NT threads:
// the vectors [kb, ke) of the tile in (c, vector) order.
template <int NT, int U, bool HOST>
__device__ __forceinline__ void copy_runs(char *d, const char *s, int64_t d_sc, int64_t s_sc,
                                          uint32_t R, int32_t C, uint32_t kb, uint32_t ke) {
    const uint32_t total = R * (uint32_t)C < ke ? R * (uint32_t)C : ke;
    for (uint32_t k0 = kb + worker_tid<NT>(); k0 < total; k0 += NT * U) {
        v4u v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t k = k0 + u * NT;
            if (k < total) {
                const uint32_t c = k >= R;
                const uint32_t w = k - c * R;
                v[u] = ld16(s + c * s_sc + (int64_t)w * 16);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t k = k0 + u * NT;
            if (k < total) {
                const uint32_t c = k >= R;
                const uint32_t w = k - c * R;
                st16<HOST>(d + c * d_sc + (int64_t)w * 16, v[u]);
            }
        }
    }
}

// Everything a tile's row loop needs, fixed for the tile.
struct Tile {
    const char *t_base;   // tiling side at (l, page, c = 0, slot = 0, h = 0)
    int32_t sa, sb;       // tiling-side slots [sa, sb) of this tile
    int32_t ntok;         // sb - sa
    // buffer other side
    const char *o_row0;   // other side at (l, c = 0, token of slot sa, h = 0)
    int64_t o_sc;         // buffer: bytes between kv components of the block
    // pool other side
    int32_t qo_a;         // other-side position of slot sa
    int32_t jo0;          // other-side logical page of qo_a
    int32_t pid;          // this lane's piece page id (-1: invalid / unused)
    int32_t l;
};

// General row-resolving copy.  Vectors are enumerated in (c, slot, h, v)
// order when the tiling side is token-major (its memory order), else in
// blocks of slots as described below, with the slots outside [sa, sb)
// masked.
template <int OP, bool TTHD, int NT, bool HOST, int U>
__device__ __forceinline__ void copy_rows(const Params &p, const Req &q, const Tile &t, uint32_t kb0,
                                          uint32_t ke) {
    constexpr bool kTileSrc = OP == OP_GATHER;
    constexpr bool kOtherBuf = OP != OP_TRANSFER;
    const Side &ts = kTileSrc ? p.src : p.dst;
    const Side &os = kTileSrc ? p.dst : p.src;
    const uint32_t H = p.H, vpr = p.vpr, row = p.row_bytes;
    // A head-major tiling side takes its vectors in (c, slot block, h, slot,
    // v) order over the blocks of SB slots that meet [sa, sb): the tiling
    // side's writes are SB-row runs, and the other side's reads, whose
    // consecutive heads are adjacent, fill whole slots within a few passes.
    // (Page order, one head at a time, left the reads 256-byte pieces a
    // kilobyte apart: 11% slower on a 16-token -> 64-token relayout.)
    constexpr uint32_t SB = KVX_SLOT_BLOCK;
    const uint32_t blk0 = (uint32_t)t.sa / SB, nblk = ((uint32_t)t.sb - 1) / SB - blk0 + 1;
    const uint32_t rows_c = TTHD ? (uint32_t)t.ntok * H : H * nblk * SB;
    const uint32_t total = rows_c * vpr * (uint32_t)p.C < ke ? rows_c * vpr * (uint32_t)p.C : ke;
    const char *o_l = os.base + (int64_t)t.l * os.s_l;
    // The trip count is the same for every lane: the page-id broadcast below
    // reads other lanes, which must all still be active.
    for (uint32_t kb = kb0; kb < total; kb += NT * U) {
        const char *src[U];
        char *dst[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t kk = kb + worker_tid<NT>() + u * NT;
            const uint32_t k = kk < total ? kk : total - 1;
            bool valid = kk < total;
            const uint32_t rw = fd_div(p.fd_vpr, k);
            const uint32_t v = k - rw * vpr;
            const uint32_t c = rw >= rows_c;
            const uint32_t rr = rw - c * rows_c;
            uint32_t h, slot;
            if (TTHD) {
                const uint32_t tt = fd_div(p.fd_H, rr);
                h = rr - tt * H;
                slot = t.sa + tt;
            } else {
                const uint32_t q1 = rr / SB;
                const uint32_t blk = fd_div(p.fd_H, q1);
                h = q1 - blk * H;
                slot = (blk0 + blk) * SB + (rr - q1 * SB);
                valid = valid && slot >= (uint32_t)t.sa && slot < (uint32_t)t.sb;
            }
            const int32_t tt = (int32_t)slot - t.sa;  // token index within the tile
            const char *ta = t.t_base + c * ts.s_c + (int64_t)slot * ts.s_t +
                             (int64_t)h * ts.s_h + v * 16;
            const char *oa;
            if (kOtherBuf) {
                oa = t.o_row0 + c * t.o_sc + (int64_t)tt * H * row + h * row + v * 16;
            } else {
                const uint32_t qo = (uint32_t)(t.qo_a + tt);
                const uint32_t jo = fd_div(p.fd_To, qo);
                const uint32_t so = qo - jo * (uint32_t)os.T;
                const uint32_t piece = jo - (uint32_t)t.jo0;
                int32_t pg = __shfl(t.pid, piece < kWave ? piece : kWave - 1, kWave);
                if (valid && piece >= kWave) {
                    // More pieces than lanes: resolve this row's page directly.
                    const int64_t idx = q.o_pt_off + jo;
                    pg = -1;
                    if (idx < 0 || idx >= os.pt_len) {
                        report(p, KVX_DERR_PT_RANGE);
                    } else {
                        const int32_t id = os.pt[idx];
                        if (id < 0 || id >= os.N) report(p, KVX_DERR_SRC_PAGE);
                        else pg = id;
                    }
                }
                valid = valid && pg >= 0;
                oa = o_l + (int64_t)pg * os.s_p + c * os.s_c + (int64_t)so * os.s_t +
                     (int64_t)h * os.s_h + v * 16;
            }
            ok[u] = valid;
            src[u] = kTileSrc ? ta : oa;
            dst[u] = const_cast<char *>(kTileSrc ? oa : ta);
        }
        v4u val[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) val[u] = ld16(src[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) st16<HOST>(dst[u], val[u]);
    }
}

// Tile (request q, its tiling-side page jj, layer l): the vectors [kb, ke) of
// the tile's vector order, U vectors per thread in flight.
template <int OP, bool TTHD, int NT, bool HOST, int UF, int UR>
__device__ __forceinline__ void do_tile(const Params &p, const Req &q, int64_t jj, int32_t layer,
                                        uint32_t kb, uint32_t ke) {
    constexpr bool kTileSrc = OP == OP_GATHER;
    constexpr bool kOtherBuf = OP != OP_TRANSFER;
    const Side &ts = kTileSrc ? p.src : p.dst;
    const Side &os = kTileSrc ? p.dst : p.src;

    Tile t;
    t.l = layer;
    const int64_t j = q.j0 + jj;
    const int64_t page_lo = j * ts.T;
    const int64_t qa = page_lo > q.t_start ? page_lo : q.t_start;
    const int64_t q_end = (int64_t)q.t_start + q.n;
    const int64_t qb = page_lo + ts.T < q_end ? page_lo + ts.T : q_end;
    t.sa = (int32_t)(qa - page_lo);
    t.sb = (int32_t)(qb - page_lo);
    t.ntok = t.sb - t.sa;

    // Tiling-side page (one per tile; a uniform load).
    const int64_t tidx = q.t_pt_off + j;
    if (tidx < 0 || tidx >= ts.pt_len) {
        if (worker_tid<NT>() == 0) report(p, KVX_DERR_PT_RANGE);
        return;
    }
    const int32_t tpage = ts.pt[tidx];
    if (tpage < 0 || tpage >= ts.N) {
        if (worker_tid<NT>() == 0) report(p, kTileSrc ? KVX_DERR_SRC_PAGE : KVX_DERR_DST_PAGE);
        return;
    }
    t.t_base = ts.base + (int64_t)t.l * ts.s_l + (int64_t)tpage * ts.s_p;

    const int64_t run_t = (int64_t)t.ntok * p.H * p.vpr;  // vectors per kv run
    if (kOtherBuf) {
        const int64_t H_row = (int64_t)p.H * p.row_bytes;
        const int64_t i0 = qa - q.t_start;
        t.o_sc = (int64_t)q.n * H_row;
        t.o_row0 = os.base + q.blk + (int64_t)t.l * p.C * t.o_sc + i0 * H_row;
        t.pid = -1;
        t.qo_a = 0;
        t.jo0 = 0;
        if (p.flat) {
            const char *tb = t.t_base + (int64_t)t.sa * ts.s_t;
            if (kTileSrc)
                copy_runs<NT, UF, HOST>(const_cast<char *>(t.o_row0), tb, t.o_sc, ts.s_c,
                                        (uint32_t)run_t, p.C, kb, ke);
            else
                copy_runs<NT, UF, HOST>(const_cast<char *>(tb), t.o_row0, ts.s_c, t.o_sc,
                                        (uint32_t)run_t, p.C, kb, ke);
            return;
        }
    } else {
        const int32_t delta = q.o_start - q.t_start;
        t.qo_a = (int32_t)qa + delta;
        t.jo0 = (int32_t)fd_div(p.fd_To, (uint32_t)t.qo_a);
        const int32_t jo1 = (int32_t)fd_div(p.fd_To, (uint32_t)((int32_t)qb - 1 + delta));
        const int32_t K = jo1 - t.jo0 + 1;
        const int32_t lane = threadIdx.x & (kWave - 1);
        t.pid = -1;
        if (lane < K) {
            const int64_t idx = q.o_pt_off + t.jo0 + lane;
            uint32_t bad = 0;
            if (idx < 0 || idx >= os.pt_len) {
                bad = KVX_DERR_PT_RANGE;
            } else {
                const int32_t id = os.pt[idx];
                if (id < 0 || id >= os.N) bad = KVX_DERR_SRC_PAGE;
                else t.pid = id;
            }
            if (bad && worker_tid<NT>() < kWave) report(p, bad);   // the worker's first wavefront
        }
        if (p.flat && K == 1) {
            const int32_t pg = __builtin_amdgcn_readfirstlane(t.pid);
            if (pg < 0) return;
            const int32_t so0 = t.qo_a - t.jo0 * os.T;
            const char *ob = os.base + (int64_t)t.l * os.s_l + (int64_t)pg * os.s_p +
                             (int64_t)so0 * os.s_t;
            const char *tb = t.t_base + (int64_t)t.sa * ts.s_t;
            copy_runs<NT, UF, HOST>(const_cast<char *>(tb), ob, ts.s_c, os.s_c, (uint32_t)run_t,
                                    p.C, kb, ke);
            return;
        }
    }
    copy_rows<OP, TTHD, NT, HOST, UR>(p, q, t, kb, ke);
}

// Inclusive sum of x over the workgroup's threads (x = 0 past the chunk).
// Every thread of the workgroup must call it: it contains barriers.
__device__ __forceinline__ int64_t block_scan(int64_t x, int64_t *s_wave) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const int64_t y = __shfl_up(x, d, kWave);
        if (lane >= d) x += y;
    }
    if (lane == kWave - 1) s_wave[wid] = x;
    __syncthreads();
    for (int w = 0; w < wid; ++w) x += s_wave[w];
    return x;
}

template <int OP, bool TTHD, int NT, bool HOST>
__global__ void __launch_bounds__(kBlock) kvx_copy_kernel(Params p) {
    constexpr int kWorkers = kBlock / NT;
    // Records are taken kBlock at a time: each thread reads one and counts
    // its tiles, a workgroup scan turns the counts into tile ranges, and the
    // workgroup's tiles inside the chunk find their record by binary search.
    __shared__ int64_t s_end[kBlock];   // end (exclusive) of record i's tiles in the chunk
    __shared__ int64_t s_wave[kBlock / kWave];
    Req q;
    int32_t cached = -1;
    const int64_t stride = (int64_t)gridDim.x * kWorkers;
    int64_t tile = (int64_t)blockIdx.x * kWorkers + threadIdx.x / NT, chunk_base = 0;
    for (int32_t r0 = 0; r0 < p.n_reqs; r0 += kBlock) {
        const int32_t nr = p.n_reqs - r0 < kBlock ? p.n_reqs - r0 : kBlock;
        int64_t cnt = 0;
        if ((int32_t)threadIdx.x < nr) {
            Req mine;
            if (!load_req<OP>(p, r0 + threadIdx.x, mine) && blockIdx.x == 0)
                report(p, KVX_DERR_BAD_REQ);
            cnt = mine.tiles;
        }
        s_end[threadIdx.x] = block_scan(cnt, s_wave);
        __syncthreads();
        const int64_t chunk_tiles = s_end[kBlock - 1];
        for (; tile < chunk_base + chunk_tiles; tile += stride) {   // uniform per worker
            const int64_t local = tile - chunk_base;
            int32_t lo = 0, hi = nr - 1;             // first record whose range ends past `local`
            while (lo < hi) {
                const int32_t mid = (lo + hi) >> 1;
                if (s_end[mid] > local) hi = mid;
                else lo = mid + 1;
            }
            if (r0 + lo != cached) {
                load_req<OP>(p, r0 + lo, q);
                cached = r0 + lo;
            }
            const int64_t in_rec = local - (lo ? s_end[lo - 1] : 0);
            const int64_t jj = in_rec / p.L;
            do_tile<OP, TTHD, NT, HOST, KVX_UNROLL_FLAT, KVX_UNROLL_ROWS>(
                p, q, jj, (int32_t)(in_rec - jj * p.L), 0u, 0xFFFFFFFFu);
        }
        chunk_base += chunk_tiles;
        __syncthreads();                             // s_end and s_wave are rewritten next chunk
    }
}

// Lane k's row of a sweep piece: kv component c, slot, head h, vector v of
// the row, in the vector order of copy_rows (a head-major destination in
// blocks of KVX_SWEEP_SLOT_BLOCK slots); valid is cleared for a masked slot
// of a head-major destination.
template <bool TTHD>
__device__ __forceinline__ void tile_row(const Params &p, uint32_t k, uint32_t rows_c, int32_t sa,
                                         int32_t sb, uint32_t blk0, uint32_t &c, uint32_t &slot,
                                         uint32_t &h, uint32_t &v, bool &valid) {
    constexpr uint32_t SB = KVX_SWEEP_SLOT_BLOCK;
    const uint32_t rw = fd_div(p.fd_vpr, k);
    v = k - rw * p.vpr;
    c = rw >= rows_c;
    const uint32_t rr = rw - c * rows_c;
    if (TTHD) {
        const uint32_t tt = fd_div(p.fd_H, rr);
        h = rr - tt * p.H;
        slot = (uint32_t)sa + tt;
    } else {
        const uint32_t q1 = rr / SB;
        const uint32_t blk = fd_div(p.fd_H, q1);
        h = q1 - blk * p.H;
        slot = (blk0 + blk) * SB + (rr - q1 * SB);
        valid = valid && slot >= (uint32_t)sa && slot < (uint32_t)sb;
    }
}

// One piece of the sweep: the vectors [kb, kb + 64) of destination page slot
// d of layer l, one vector per lane, in the vector order of copy_rows (a
// head-major destination in blocks of KVX_SWEEP_SLOT_BLOCK slots, the slots
// outside the page's range masked).  Every load of metadata on the path that copies (the slot,
// the destination page id, and the source page id when all the piece's rows
// lie in one source page, the usual case) is uniform and comes before the
// first store or atomic, so it goes through the scalar cache.  FLAT (both
// sides token-major with every head): the page is C runs of contiguous
// vectors on both sides, each lane finds its token's source page, and a
// piece whose rows lie in one source page is a plain vector copy.  Errors
// are reported for the positions the piece covers, destination first.  The
// slot's fields are only trusted as far as keeping every access inside the
// pools and tables; whether they match the records is checked separately
// (slot_agrees).
template <bool TTHD, bool FLAT, bool HOST>
__device__ __forceinline__ void sweep_piece(const Params &p, const kvx_plan_slot &d, uint32_t l,
                                            uint32_t kb) {
    const Side &ts = p.dst, &os = p.src;
    const int32_t sa = d.dst_slot, so_a = d.src_slot;
    const uint32_t ntok = (uint32_t)d.n_tokens;
    if (!((uint32_t)sa < (uint32_t)ts.T && ntok - 1u < (uint32_t)(ts.T - sa) &&
          (uint32_t)so_a < (uint32_t)os.T))
        return;
    const int32_t sb = sa + (int32_t)ntok;
    constexpr uint32_t SB = KVX_SWEEP_SLOT_BLOCK;
    const uint32_t blk0 = (uint32_t)sa / SB, nblk = ((uint32_t)sb - 1) / SB - blk0 + 1;
    const uint32_t rows_c = TTHD ? ntok * p.H : p.H * nblk * SB;
    const uint32_t total = rows_c * p.vpr * (uint32_t)p.C;
    if (kb >= total) return;
    const uint32_t lane = threadIdx.x;
    const uint32_t k = kb + lane;
    bool valid = k < total;

    // per lane: the row (FLAT: kv component and vector of the run) and its
    // source page, counted from the slot's; jo0 is that of the first live lane
    uint32_t c = 0, slot = 0, h = 0, v = 0, jo, jo0, w = 0;
    if (FLAT) {
        const uint32_t R = ntok * p.H * p.vpr;                 // vectors per kv run
        const uint32_t kc = valid ? k : kb;
        c = kc >= R;
        w = kc - c * R;
        jo = fd_div(p.fd_To, (uint32_t)so_a + fd_div(p.fd_hv, w));
        jo0 = __builtin_amdgcn_readfirstlane(jo);              // lane 0 is live
    } else {
        tile_row<TTHD>(p, valid ? k : total - 1, rows_c, sa, sb, blk0, c, slot, h, v, valid);
        const uint64_t live = __ballot(valid);
        if (live == 0) return;
        jo = fd_div(p.fd_To, (uint32_t)so_a + (slot - (uint32_t)sa));
        jo0 = __builtin_amdgcn_readlane(jo, __builtin_ctzll(live));
    }
    const bool one = __ballot(valid && jo != jo0) == 0;
    // The sweep runs only on tables of at most INT32_MAX entries, so 32-bit
    // unsigned compares also reject negative indices (jo0 < 2^21 cannot
    // carry a non-negative src_idx past 2^32).
    const bool t_in = (uint32_t)d.dst_idx < (uint32_t)ts.pt_len;
    const uint32_t oidx0 = (uint32_t)d.src_idx + jo0;
    const bool o_in = d.src_idx >= 0 && oidx0 < (uint32_t)os.pt_len;
    // both page ids are read before any error is reported (an atomic ahead
    // of them would turn them into vector loads)
    const int32_t tpage = t_in ? cload(ts.pt + (uint32_t)d.dst_idx) : -1;
    const int32_t opage0 = t_in && one && o_in ? cload(os.pt + oidx0) : -1;
    const bool pages_ok = (uint32_t)tpage < (uint32_t)ts.N && (uint32_t)opage0 < (uint32_t)os.N;
    char *t_base = ts.base + (int64_t)l * ts.s_l + (int64_t)tpage * ts.s_p;
    const char *o_l = os.base + (int64_t)l * os.s_l;
    if (FLAT && one && pages_ok) {
        // the usual case: the piece's rows in one source page, both pages valid
        if (!valid) return;
        // source slot of the page's first token, counted from source page jo0
        const int64_t so = (int64_t)so_a - (int64_t)jo0 * os.T;
        const char *s = o_l + (int64_t)opage0 * os.s_p + so * os.s_t;
        char *dd = t_base + (int64_t)sa * ts.s_t;
        st16<HOST>(dd + c * ts.s_c + (int64_t)w * 16, ld16(s + c * os.s_c + (int64_t)w * 16));
        return;
    }
    // errors of the page and of a single source page, destination first
    if (!t_in || (uint32_t)tpage >= (uint32_t)ts.N) {
        if (lane == 0) report(p, t_in ? KVX_DERR_DST_PAGE : KVX_DERR_PT_RANGE);
        return;
    }
    if (one && !pages_ok) {
        if (lane == 0) report(p, o_in ? KVX_DERR_SRC_PAGE : KVX_DERR_PT_RANGE);
        return;
    }
    if (FLAT) {                     // rows in two source pages: resolve them as the general case
        tile_row<true>(p, valid ? k : total - 1, rows_c, sa, sb, blk0, c, slot, h, v, valid);
        jo = fd_div(p.fd_To, (uint32_t)so_a + (slot - (uint32_t)sa));
    }
    int32_t pg = one ? opage0 : -1;
    if (!one && valid) {
        const int64_t idx = (int64_t)d.src_idx + jo;
        if (idx < 0 || idx >= os.pt_len) {
            report(p, KVX_DERR_PT_RANGE);
        } else {
            const int32_t id = os.pt[idx];
            if (id < 0 || id >= os.N) report(p, KVX_DERR_SRC_PAGE);
            else pg = id;
        }
    }
    if (!valid || pg < 0) return;
    const uint32_t so = (uint32_t)so_a + (slot - (uint32_t)sa) - jo * (uint32_t)os.T;
    const char *src = o_l + (int64_t)pg * os.s_p + c * os.s_c + (int64_t)so * os.s_t +
                      (int64_t)h * os.s_h + v * 16;
    char *dst = t_base + c * ts.s_c + (int64_t)slot * ts.s_t + (int64_t)h * ts.s_h + v * 16;
    st16<HOST>(dst, ld16(src));
}

__device__ __forceinline__ int32_t clamp_i32(int64_t x) {
    return x < INT32_MIN ? INT32_MIN : x > INT32_MAX ? INT32_MAX : (int32_t)x;
}

// Whether slot d of the plan is page qi of the plan the records imply: its
// record's prefix range holds qi, and its fields are those of that record's
// page qi - prefix[r].  Run once per slot (by one workgroup of layer 0).
__device__ __forceinline__ bool slot_agrees(const Params &p, int64_t qi, const kvx_plan_slot &d) {
    const int32_t r = d.req;
    if (r < 0 || r >= p.n_reqs) return false;
    Req q;
    if (!load_req<OP_TRANSFER>(p, r, q)) return false;
    const int64_t jj = qi - p.prefix[r];
    if (jj < 0 || qi >= p.prefix[r + 1] || jj >= q.pages) return false;
    const int64_t j = (int64_t)q.j0 + jj, page_lo = j * p.dst.T;
    const int64_t q_end = (int64_t)q.t_start + q.n;
    const int64_t qa = page_lo > q.t_start ? page_lo : q.t_start;
    const int64_t qb = page_lo + p.dst.T < q_end ? page_lo + p.dst.T : q_end;
    const int64_t pos = qa - q.t_start + q.o_start;
    const int64_t jo = pos / p.src.T;
    return d.dst_idx == clamp_i32(q.t_pt_off + j) && d.src_idx == clamp_i32(q.o_pt_off + jo) &&
           d.dst_slot == (int32_t)(qa - page_lo) && d.n_tokens == (int32_t)(qb - qa) &&
           d.src_slot == (int32_t)(pos - jo * p.src.T);
}

// Page slot qi of layer l: read its slot, copy the workgroup's
// KVX_SWEEP_PIECES pieces one after the other, and (one workgroup per slot)
// check the slot against the records.
template <bool TTHD, bool FLAT, bool HOST>
__device__ __forceinline__ void sweep_slot(const Params &p, int64_t qi, uint32_t l, uint32_t part) {
    const kvx_plan_slot d = cload(p.slots + qi);
    const uint32_t piece0 = part * KVX_SWEEP_PIECES;
#pragma unroll
    for (uint32_t i = 0; i < KVX_SWEEP_PIECES; ++i)
        sweep_piece<TTHD, FLAT, HOST>(p, d, l, (piece0 + i) * kWave);
    if (l == 0 && part == 0 && !slot_agrees(p, qi, d) && threadIdx.x == 0) report(p, KVX_DERR_BAD_PLAN);
}

// Sweep kernel (a planned pool -> pool transfer): one wavefront per
// workgroup, and workgroup b copies one piece of 64 vectors (1 KiB) of one
// destination page of one layer in each pass, found by one read of the
// plan.  Workgroups are numbered layer by layer and page slot by page slot
// within a layer (pages in plan order), so the hardware dispatcher, which
// starts them in order, keeps the pieces in flight on the whole GPU inside a
// small window that slides through the transfer.  (A persistent grid lets
// its workers drift over the whole transfer; on the same pools this order
// moves up to 16% more bytes per second for 256 KiB pages.)  The dispatcher
// deals consecutive workgroups to the 8 XCDs in turn, so within each group
// of 8 page slots the numbering gives XCD x every piece of slot x, in order:
// each page is copied by one XCD.  (Measured on the same pools: 1.5-3% more
// bytes per second than pieces dealt across the XCDs for 72 and 256 KiB
// pages, 6% for 128 KiB pages; a contiguous eighth of every page per XCD
// is 10% slower.)  The launch has layers x sweep_pages x ppt workgroups,
// with sweep_pages about plan_pages / KVX_SWEEP_PASSES (fewer when the grid
// is capped): each workgroup goes on to the slots sweep_pages apart, up to
// plan_pages.  The first slot is taken outside that loop, so that its loads
// precede every store of the kernel.  Workgroup 0 finally checks the prefix
// against the records and plan_pages, and reports malformed records.
template <bool TTHD, bool FLAT, bool HOST>
__global__ void __launch_bounds__(kWave) kvx_sweep_kernel(Params p) {
    const uint32_t b = blockIdx.x;
    uint32_t slot = fd_div(p.fd_ppt, b);                       // (layer, page slot)
    uint32_t part = b - slot * p.sweep_ppt;
    {
        // In each whole group of 8 page slots, XCD b % 8 takes slot 8g + b % 8
        // (its pieces in order): every page is copied by one XCD.
        const uint32_t g = slot >> 3;
        if ((g << 3) + 8u <= (uint32_t)p.L * (uint32_t)p.sweep_pages) {
            const uint32_t r = b - (g << 3) * p.sweep_ppt;
            slot = (g << 3) + (r & 7u);
            part = r >> 3;
        }
    }
    const uint32_t l = fd_div(p.fd_sp, slot);
    const int64_t q0 = (int64_t)(slot - l * (uint32_t)p.sweep_pages);
    sweep_slot<TTHD, FLAT, HOST>(p, q0, l, part);
    for (int64_t qi = q0 + p.sweep_pages; qi < p.plan_pages; qi += p.sweep_pages)  // later passes
        sweep_slot<TTHD, FLAT, HOST>(p, qi, l, part);
    if (b == 0) {
        // prefix[0] = 0, prefix[r + 1] - prefix[r] = pages of record r, and
        // prefix[n_reqs] = plan_pages
        bool bad_plan = p.prefix[0] != 0 || p.prefix[p.n_reqs] != p.plan_pages;
        for (int32_t r0 = 0; r0 < p.n_reqs; r0 += kWave) {
            const int32_t r = r0 + (int32_t)threadIdx.x;
            if (r < p.n_reqs) {
                Req mine;
                if (!load_req<OP_TRANSFER>(p, r, mine)) report(p, KVX_DERR_BAD_REQ);
                bad_plan = bad_plan || p.prefix[r + 1] - p.prefix[r] != mine.pages;
            }
        }
        if (bad_plan) report(p, KVX_DERR_BAD_PLAN);
    }
}

typedef void (*KernelFn)(Params);

constexpr int kFlatNT = KVX_FLAT_WAVE_TILES ? kWave : kBlock;
constexpr int kRowsNT = KVX_ROWS_WAVE_TILES ? kWave : kBlock;

template <int OP, bool HOST>
KernelFn pick_op(bool tthd, bool flat) {
    if (flat)
        return tthd ? kvx_copy_kernel<OP, true, kFlatNT, HOST>
                    : kvx_copy_kernel<OP, false, kFlatNT, HOST>;
    return tthd ? kvx_copy_kernel<OP, true, kRowsNT, HOST> : kvx_copy_kernel<OP, false, kRowsNT, HOST>;
}

KernelFn pick(int op, bool tthd, bool flat, bool host) {
    switch (op) {
    case OP_TRANSFER:
        return host ? pick_op<OP_TRANSFER, true>(tthd, flat) : pick_op<OP_TRANSFER, false>(tthd, flat);
    case OP_GATHER:
        return host ? pick_op<OP_GATHER, true>(tthd, flat) : pick_op<OP_GATHER, false>(tthd, flat);
    default:
        return host ? pick_op<OP_SCATTER, true>(tthd, flat) : pick_op<OP_SCATTER, false>(tthd, flat);
    }
}

}  // namespace

// Sweep grid when the host chose it (p.sweep), else a persistent grid: as
// many workgroups as the device holds at once.
int launch(const Params &p, hipStream_t stream) {
    if (p.sweep) {
        KernelFn fs;
        if (p.flat)
            fs = p.dst_host ? kvx_sweep_kernel<true, true, true> : kvx_sweep_kernel<true, true, false>;
        else if (p.dst.tok_contig)
            fs = p.dst_host ? kvx_sweep_kernel<true, false, true> : kvx_sweep_kernel<true, false, false>;
        else
            fs = p.dst_host ? kvx_sweep_kernel<false, false, true> : kvx_sweep_kernel<false, false, false>;
        const uint64_t blocks = (uint64_t)p.L * (uint64_t)p.sweep_pages * p.sweep_ppt;
        hipLaunchKernelGGL(fs, dim3((uint32_t)blocks), dim3(kWave), 0, stream, p);
        return hipGetLastError();
    }
    const bool tthd = (p.op == OP_GATHER ? p.src : p.dst).tok_contig != 0;
    KernelFn fn = pick(p.op, tthd, p.flat != 0, p.dst_host != 0);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    int per_cu = p.flat ? KVX_BLOCKS_PER_CU : KVX_ROWS_BLOCKS_PER_CU;
    if (per_cu <= 0) {
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(fn),
                                                         kBlock, 0);
        if (e != hipSuccess) return e;
        if (per_cu < 1) per_cu = 1;
    }
    hipLaunchKernelGGL(fn, dim3(cus * per_cu), dim3(kBlock), 0, stream, p);
    return hipGetLastError();
}

}  // namespace kvx
