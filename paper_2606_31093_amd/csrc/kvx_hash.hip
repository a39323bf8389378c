// kvx_hash.hip -- chained page hashes for gfx950 (Omni-Flow Sec. 5.1:
// each page's hash encodes its predecessor's, so equal hashes mean an equal
// prefix page by page).  Definition, with fnv = FNV-1a 64:
//   c_j = fnv(records of page j),   h_j = fnv(le64(h_{j-1}) || le64(c_j)).
//
// One wavefront per request (a grid-stride loop over requests).  Pages are
// taken 64 at a time: lane j computes the digest of page j of the chunk,
// issuing the loads of 64 words (a whole 256-byte page of token ids) before
// hashing them, so the cache lines a page shares with its neighbours are
// fetched while they are all in flight rather than once per batch.  The
// chain then runs through the chunk's digests in page order, each broadcast
// from its lane, and lane j keeps h_j, so the chunk's hashes leave in one
// coalesced store.  Nothing is allocated.

#include "kvx_hash.h"

namespace kvx {
namespace {

constexpr int kWave = 64;
#ifndef KVX_HASH_BATCH
#define KVX_HASH_BATCH 64   // words in flight per lane (measured: 16, 32, 64)
#endif
constexpr uint64_t kBasis = 0xcbf29ce484222325ull;
constexpr uint64_t kPrime = 0x100000001b3ull;

__device__ __forceinline__ uint64_t fnv_word(uint64_t h, uint32_t w) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        h ^= (w >> (8 * b)) & 0xffu;
        h *= kPrime;
    }
    return h;
}

__device__ __forceinline__ uint64_t fnv_u64(uint64_t h, uint64_t v) {
    h = fnv_word(h, (uint32_t)v);
    return fnv_word(h, (uint32_t)(v >> 32));
}

// FNV-1a of nw 32-bit words, KVX_HASH_BATCH loads in flight.
__device__ __forceinline__ uint64_t digest(const uint32_t *w, int64_t nw) {
    constexpr int B = KVX_HASH_BATCH;
    uint64_t c = kBasis;
    int64_t i = 0;
    for (; i + B <= nw; i += B) {
        uint32_t v[B];
#pragma unroll
        for (int u = 0; u < B; ++u) v[u] = w[i + u];
#pragma unroll
        for (int u = 0; u < B; ++u) c = fnv_word(c, v[u]);
    }
    for (; i < nw; ++i) c = fnv_word(c, w[i]);
    return c;
}

__device__ __forceinline__ uint64_t lane_u64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

__global__ void __launch_bounds__(kWave) kvx_page_hash_kernel(HashParams p) {
    const int lane = threadIdx.x;
    const int64_t wpr = p.rec_bytes / 4;
    for (int32_t r = blockIdx.x; r < p.n_reqs; r += gridDim.x) {
        const kvx_hash_req &q = p.reqs[r];
        const int64_t off = q.payload_off, out_off = q.out_off;
        const int32_t n = q.n_positions;
        const int64_t pages = n > 0 ? ((int64_t)n + p.T - 1) / p.T : 0;
        const bool ok = n >= 0 && q.reserved == 0 && off >= 0 && off <= p.payload_positions - n &&
                        out_off >= 0 && out_off <= p.out_len - pages;
        if (!ok) {
            if (lane == 0 && p.err) atomicOr(p.err, KVX_DERR_BAD_REQ);
            continue;                       // uniform across the wavefront
        }
        uint64_t h = q.seed;                // uniform chain state
        for (int64_t j0 = 0; j0 < pages; j0 += kWave) {
            const int in_chunk = pages - j0 < kWave ? (int)(pages - j0) : kWave;
            const int64_t j = j0 + lane;
            uint64_t c = 0;
            if (lane < in_chunk) {
                const int64_t first = j * p.T;
                const int64_t count = n - first < p.T ? n - first : p.T;
                c = digest(p.payload + (off + first) * wpr, count * wpr);
            }
            uint64_t mine = 0;
            for (int k = 0; k < in_chunk; ++k) {
                h = fnv_u64(fnv_u64(kBasis, h), lane_u64(c, k));
                if (lane == k) mine = h;
            }
            if (lane < in_chunk) p.out[out_off + j] = mine;
        }
    }
}

}  // namespace

int launch_hash(const HashParams &p, hipStream_t stream) {
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int grid = p.n_reqs < cus * 32 ? p.n_reqs : cus * 32;
    hipLaunchKernelGGL(kvx_page_hash_kernel, dim3(grid), dim3(kWave), 0, stream, p);
    return hipGetLastError();
}

}  // namespace kvx
