// kvx_internal.h -- launch parameters shared by the C-ABI layer and the HIP
// kernels of libkvx.  Not part of the public interface (include/kvx.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvx.h"

namespace kvx {

// Unsigned division by a divisor fixed for a launch, for dividends below
// 2^31: q = floor(n * m / 2^(31 + l)) with l = ceil(log2 d) and
// m = ceil(2^(31 + l) / d).  Exact because m * d - 2^(31 + l) < d <= 2^l,
// so the error term n * (m * d - 2^(31 + l)) / 2^(31 + l) stays below
// n / 2^31 < 1 / d of one quotient step (Granlund and Montgomery,
// "Division by invariant integers using multiplication", PLDI 1994).
struct FastDiv {
    uint32_t d;  // divisor, 1 <= d < 2^31
    uint32_t m;  // multiplier (unused when d == 1)
    uint32_t s;  // post-shift l - 1
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f{d, 0u, 0u};
    if (d > 1) {
        uint32_t l = 0;
        while ((1ull << l) < d) ++l;
        f.m = (uint32_t)(((1ull << (31 + l)) + d - 1) / d);
        f.s = l - 1;
    }
    return f;
}

__host__ __device__ inline uint32_t fd_div(const FastDiv &f, uint32_t n) {
    return f.d == 1 ? n : (uint32_t)(((uint64_t)n * f.m) >> 32) >> f.s;
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
};

// Launch on `stream`; returns a hipError_t value.
int launch(const Params &p, hipStream_t stream);

}  // namespace kvx
