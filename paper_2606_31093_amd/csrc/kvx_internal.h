// kvx_internal.h -- launch parameters shared by the C-ABI layer and the HIP
// kernels of libkvx.  Not part of the public interface (include/kvx.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvx.h"

#ifndef KVX_SLOT_BLOCK
#define KVX_SLOT_BLOCK 2  // head-major tiling: slots per block of the vector order (measured best)
#endif
// The same for the sweep into a head-major destination (measured: 16 moves
// the relayout 1.4% faster than 2, 8 and 64 in between; the persistent grid
// loses 3% with blocks of 8).
#ifndef KVX_SWEEP_SLOT_BLOCK
#define KVX_SWEEP_SLOT_BLOCK 16
#endif
// A planned transfer sweeps when its records copy at least this many bytes
// per destination page and layer on average (measured: from 72 KiB pages up
// the sweep holds its rate in every placement of the pools, where the
// persistent grid's varies by up to 20% between processes).
#ifndef KVX_SWEEP_MIN_BYTES
#define KVX_SWEEP_MIN_BYTES (64 << 10)
#endif
// Pieces of 64 vectors one sweep workgroup copies, one after the other.
#ifndef KVX_SWEEP_PIECES
#define KVX_SWEEP_PIECES 1
#endif
// Passes of a sweep launch over the plan's pages: each workgroup copies its
// piece of one page in each pass, pages plan_pages / passes apart.  Measured:
// 3 passes move 128-256 KiB pages 4-6% faster than 1; 2 passes beat 3 by
// 0.5-1.5% at every page size tried from 64 to 108 KiB, where from 121 KiB
// copied per page and layer on average up they vary from -4% to +1%.  So
// below 96 KiB on average a launch takes 2.
#ifndef KVX_SWEEP_PASSES
#define KVX_SWEEP_PASSES 3
#endif
#ifndef KVX_SWEEP_SMALL_BYTES
#define KVX_SWEEP_SMALL_BYTES (96 << 10)
#endif
#ifndef KVX_SWEEP_PASSES_SMALL
#define KVX_SWEEP_PASSES_SMALL 2
#endif
// Most workgroups of one sweep launch: the work-items of a launch (64 per
// workgroup) must stay below 2^32, and this keeps them below 2^31.  Beyond
// it, workgroups loop over page slots.
#ifndef KVX_SWEEP_MAX_BLOCKS
#define KVX_SWEEP_MAX_BLOCKS (INT32_MAX / 64)
#endif

namespace kvx {

// Unsigned division by a divisor fixed for a launch, for dividends below
// 2^31: q = floor(n * m / 2^(31 + l)) with l = ceil(log2 d) and
// m = ceil(2^(31 + l) / d).  Exact because m * d - 2^(31 + l) < d <= 2^l,
// so the error term n * (m * d - 2^(31 + l)) / 2^(31 + l) stays below
// n / 2^31 < 1 / d of one quotient step (Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994).
struct FastDiv {
    uint32_t d;   // divisor, 1 <= d < 2^31
    uint32_t m;   // ceil(2^(31 + l) / d), l = ceil(log2 d); below 2^32
    uint32_t sh;  // 31 + l
};

inline FastDiv make_fastdiv(uint32_t d) {
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    return FastDiv{d, (uint32_t)(((1ull << (31 + l)) + d - 1) / d), 31 + l};
}

// n / d for n < 2^31 without a branch: n * m / 2^(31 + l) = n / d + n * (m *
// d - 2^(31 + l)) / (d * 2^(31 + l)), and the second term, below n / 2^(31 +
// l) < 2^-l <= 1 / d, cannot reach the next multiple of 1 / d.
__host__ __device__ inline uint32_t fd_div(const FastDiv &f, uint32_t n) {
    return (uint32_t)(((uint64_t)n * f.m) >> f.sh);
}

// One side of a copy.  A pool side addresses row (l, page, c, slot, h) at
// base + l*s_l + page*s_p + c*s_c + slot*s_t + h*s_h (bytes), with base
// already moved to the first layer, kv component and head the call copies;
// a buffer side addresses row (l, c, i, h) of a request's block at
// base + blk + ((l*C + c)*n + i)*H*row + h*row, with blk the block's byte
// offset.
struct Side {
    char *base;
    int64_t s_l, s_p, s_c, s_t, s_h;
    const int32_t *pt;
    int64_t pt_len;
    int32_t T;        // tokens per page (pool side)
    int32_t N;        // pages (pool side)
    int32_t tok_contig;  // rows of consecutive slots, all copied heads, are adjacent
    int64_t cap_bytes;   // buffer side: bytes addressable from base
};

enum Op : int32_t { OP_TRANSFER = 0, OP_GATHER = 1, OP_SCATTER = 2 };

struct Params {
    Side src, dst;
    const kvx_req *reqs;
    uint32_t *err;
    int32_t n_reqs;
    int32_t op;
    int32_t L, C, H;     // layers, kv components and heads copied
    int32_t row_bytes;   // head_dim * elem_bytes, a multiple of 16
    int32_t vpr;         // 16-byte vectors per row
    int32_t elem_bytes;
    int32_t flat;        // both sides tok_contig: a tile is C contiguous runs per piece
    int32_t dst_host;    // the destination is pinned host memory (plain stores)
    FastDiv fd_vpr, fd_H, fd_To;
    FastDiv fd_Tt;       // tiling side's page_tokens
    // Sweep launch (a planned pool -> pool transfer): one workgroup per piece
    // of 64 vectors of one destination page of one layer and pass.
    // sweep_pages page slots per layer are launched (plan_pages / passes, or
    // fewer when the grid is capped; workgroups go on to the slots
    // sweep_pages apart), sweep_ppt pieces per page.  prefix[r] =
    // destination pages of records 0..r-1, slots[q] = page q of the plan.
    // sweep == 0: persistent grid.
    int32_t sweep;
    int32_t sweep_pages;
    uint32_t sweep_ppt;
    int64_t plan_pages;
    FastDiv fd_ppt, fd_sp;
    FastDiv fd_hv;       // H * vpr: vectors per token of a token-major side
    const int64_t *prefix;
    const kvx_plan_slot *slots;
};

// Launch on `stream`; returns a hipError_t value.
int launch(const Params &p, hipStream_t stream);

}  // namespace kvx
